"""Pins for the oracle's LET (Eq.3), block step (Eq.1/Eq.4, Algorithm 1),
straight-through gradients and AdamW update."""
import json
import os

import numpy as np
import pytest
import torch

from oracle.adamw import adamw
from oracle.block import block_step, fp_target
from oracle.let import let_bias, let_fold, let_init, let_w, let_x
from oracle.quant import lwc_fwd
from oracle.surrogate import freeze, surrogate_loss

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))


# ---------------------------------------------------------------- LET, Eq.3
def test_let_identity_at_unit_scale_zero_shift():
    rng = np.random.default_rng(0)
    X = rng.standard_normal((16, 32)).astype(np.float32)
    W = rng.standard_normal((8, 32)).astype(np.float32)
    B = rng.standard_normal(8).astype(np.float32)
    one, zero = np.ones(32, np.float32), np.zeros(32, np.float32)
    assert np.array_equal(let_x(X, one, zero), X)
    Wt, Bt = let_fold(W, B, one, zero)
    assert np.array_equal(Wt, W) and np.array_equal(Bt, B)


def test_let_fold_identity():
    """(X - delta)/s . (s W) + (B + delta W) = X W + B (Eq.3), in fp64 and fp32."""
    rng = np.random.default_rng(1)
    X = rng.standard_normal((64, 48)) * 3
    W = rng.standard_normal((24, 48))
    B = rng.standard_normal(24)
    s = rng.uniform(0.2, 5.0, 48)
    d = rng.standard_normal(48)
    ref = X @ W.T + B
    Xt = let_x(X, s, d, ft=np.float64)
    Wt, Bt = let_fold(W, B, s, d, ft=np.float64)
    np.testing.assert_allclose(Xt @ Wt.T + Bt, ref, rtol=1e-12, atol=1e-12)
    Xt = let_x(X, s, d).astype(np.float64)
    Wt, Bt = let_fold(W, B, s, d)
    err = np.max(np.abs(Xt @ Wt.T.astype(np.float64) + Bt - ref)) / np.max(np.abs(ref))
    assert err < 1e-5
    # wrong sign of the shift or an inverted scale breaks the identity
    Wbad, Bbad = let_w(W, 1.0 / s, np.float64), let_bias(W, B, -d, np.float64)
    assert np.max(np.abs(Xt @ Wbad.T + Bt - ref)) > 1e-2
    assert np.max(np.abs(Xt @ Wt.T + Bbad - ref)) > 1e-2


def test_let_init_worked_example():
    c = GOLD["let_init"]
    s, d = let_init(np.array(c["x"], np.float32), [np.array(c["w"], np.float32)])
    np.testing.assert_allclose(s, c["s"], rtol=1e-7)
    np.testing.assert_array_equal(d, np.float32(c["delta"]))


def test_let_init_takes_max_over_all_site_linears():
    X = np.array([[4.0, 1.0]], np.float32)
    s, _ = let_init(X, [np.array([[1.0, 1.0]], np.float32), np.array([[16.0, 0.25]], np.float32)])
    np.testing.assert_allclose(s, [0.5, 1.0], rtol=1e-7)


# ---------------------------------------------------------------- block step
def _tiny_desc(T=8, c_in=32, c_out=8, g=8, bits=3, let=False, act=16, n_lin=1, bf16=False):
    return dict(T=T, bf16=bf16, sites=[dict(width=c_in, let=let, act_bits=act)],
                linears=[dict(site=0, c_out=c_out, bits=bits, group=g) for _ in range(n_lin)])


def _tiny_params(desc, rng, bias=False):
    T = desc["T"]
    X, W, B, gl, bl, Y = [], [], [], [], [], []
    for k, s in enumerate(desc["sites"]):
        X.append(rng.standard_normal((T, s["width"])).astype(np.float32))
    for l in desc["linears"]:
        c_in = desc["sites"][l["site"]]["width"]
        W.append((rng.standard_normal((l["c_out"], c_in)) * 0.5).astype(np.float32))
        B.append(rng.standard_normal(l["c_out"]).astype(np.float32) if bias else None)
        ng = c_in // l["group"]
        gl.append(rng.uniform(1.0, 4.0, (l["c_out"], ng)))
        bl.append(rng.uniform(1.0, 4.0, (l["c_out"], ng)))
        Y.append((X[l["site"]] @ W[-1].T + rng.standard_normal((T, l["c_out"])) * 0.05).astype(np.float32))
    s = [rng.uniform(0.5, 2.0, site["width"]).astype(np.float32) if site["let"] else None
         for site in desc["sites"]]
    d = [(rng.standard_normal(site["width"]) * 0.3).astype(np.float32) if site["let"] else None
         for site in desc["sites"]]
    return X, Y, dict(W=W, B=B, gamma_logit=gl, beta_logit=bl, s=s, delta=d)


def test_block_tiny_worked_loss():
    c = GOLD["block_tiny"]
    desc = _tiny_desc(T=3, c_in=2, c_out=1, g=2, bits=2)
    params = dict(W=[np.array(c["w"], np.float32)], B=[None], gamma_logit=[np.full((1, 1), 30.0)],
                  beta_logit=[np.full((1, 1), 30.0)], s=[None], delta=[None])
    loss, out = block_step(desc, [np.array(c["x"], np.float32)], [np.array(c["y_fp"], np.float32)], params)
    np.testing.assert_allclose(loss, c["loss"][0] / c["loss"][1], rtol=1e-6)
    np.testing.assert_allclose(np.sum(out["row_loss"][0]) / 3, loss, rtol=1e-12)


def test_on_grid_weights_give_zero_loss_and_grads():
    """A weight that already lies on its own min-max grid quantises to itself,
    so the quantised block equals the full-precision block."""
    rng = np.random.default_rng(2)
    desc = _tiny_desc(T=16, c_in=64, c_out=16, g=16, bits=3)
    codes = rng.integers(0, 8, (16, 64)).astype(np.float32)
    codes[:, ::16] = 0
    codes[:, 1::16] = 7                      # every group spans the full code range
    W = (codes - 3.0) * np.float32(0.125)    # z = 3, h = 1/8: exact in fp32
    X = [rng.standard_normal((16, 64)).astype(np.float32)]
    Y = [(X[0].astype(np.float64) @ W.T.astype(np.float64)).astype(np.float32)]
    params = dict(W=[W], B=[None], gamma_logit=[np.full((16, 4), 30.0)],
                  beta_logit=[np.full((16, 4), 30.0)], s=[None], delta=[None])
    st = lwc_fwd(W, params["gamma_logit"][0], params["beta_logit"][0], 3, 16)
    np.testing.assert_array_equal(st["W_dq"], W)
    loss, out = block_step(desc, X, Y, params)
    assert loss == 0.0
    assert np.all(out["d_gamma_logit"][0] == 0) and np.all(out["d_beta_logit"][0] == 0)


def test_row_decomposition_of_lwc_only_step():
    """Without LET the loss and every clipping gradient of output row o depend
    only on row o: the step on a row subset reproduces those rows."""
    rng = np.random.default_rng(3)
    desc = _tiny_desc(T=12, c_in=32, c_out=10, g=8, bits=3)
    X, Y, p = _tiny_params(desc, rng)
    loss, out = block_step(desc, X, Y, p)
    rows = [1, 4, 9]
    d2 = _tiny_desc(T=12, c_in=32, c_out=3, g=8, bits=3)
    p2 = dict(W=[p["W"][0][rows]], B=[None], gamma_logit=[p["gamma_logit"][0][rows]],
              beta_logit=[p["beta_logit"][0][rows]], s=[None], delta=[None])
    _, out2 = block_step(d2, X, [Y[0][:, rows]], p2)
    # d2's mean runs over 3 channels instead of 10: rescale
    np.testing.assert_allclose(out2["d_gamma_logit"][0] * 3 / 10, out["d_gamma_logit"][0][rows], rtol=1e-5)
    np.testing.assert_allclose(out2["row_loss"][0], out["row_loss"][0][rows], rtol=1e-12)
    # with the whole linear's normaliser the subset reproduces the rows directly
    d3 = _tiny_desc(T=12, c_in=32, c_out=3, g=8, bits=3)
    d3["linears"][0]["mean_rows"] = 10
    _, out3 = block_step(d3, X, [Y[0][:, rows]], p2)
    np.testing.assert_allclose(out3["d_gamma_logit"][0], out["d_gamma_logit"][0][rows], rtol=1e-12)
    np.testing.assert_allclose(out3["d_beta_logit"][0], out["d_beta_logit"][0][rows], rtol=1e-12)


@pytest.mark.parametrize("let,act,bf16", [(False, 16, True), (False, 16, False), (True, 4, True)])
def test_token_decomposition_of_the_step(let, act, bf16):
    """Every term of the step is a sum over tokens for fixed parameters (the
    per-token quantiser reads only its own row), so the step over token
    chunks, each normalised by the whole token count, adds up to the step
    over all tokens: loss, row losses and every parameter gradient.  This is
    what lets the full-size checks run the oracle chunk by chunk."""
    rng = np.random.default_rng(5 + int(let) + 2 * int(bf16))
    T, n_chunks = 24, 3
    desc = _tiny_desc(T=T, c_in=32, c_out=10, g=8, bits=3, let=let, act=act, n_lin=2, bf16=bf16)
    X, Y, p = _tiny_params(desc, rng, bias=let)
    loss, out = block_step(desc, X, Y, p)
    step = T // n_chunks
    tot_loss = 0.0
    acc = None
    for c in range(n_chunks):
        dc = _tiny_desc(T=step, c_in=32, c_out=10, g=8, bits=3, let=let, act=act, n_lin=2, bf16=bf16)
        for lin in dc["linears"]:
            lin["mean_rows"] = lin["c_out"] * n_chunks
        sl = slice(c * step, (c + 1) * step)
        lc, oc = block_step(dc, [x[sl] for x in X], [y[sl] for y in Y], p)
        tot_loss += lc
        part = {k: [None if a is None else np.asarray(a, np.float64) for a in oc[k]]
                for k in ("d_gamma_logit", "d_beta_logit", "d_s", "d_delta", "row_loss")}
        if acc is None:
            acc = part
        else:
            for k in acc:
                acc[k] = [None if a is None else a + b for a, b in zip(acc[k], part[k])]
    np.testing.assert_allclose(tot_loss, loss, rtol=1e-12)
    for k in acc:
        for a, b in zip(acc[k], out[k]):
            if b is None:
                assert a is None
            else:
                np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-12 * np.max(np.abs(b)))


# ---------------------------------------------------------------- straight-through gradients
FD_CASES = [
    dict(bits=2, g=8), dict(bits=3, g=8), dict(bits=4, g=8),
    dict(bits=3, g=32),                                    # per-channel
    dict(bits=4, g=8, let=True),                           # LET without act quant
    dict(bits=4, g=8, let=True, act=4),                    # LET + per-token act quant
    dict(bits=3, g=16, let=True, act=3, n_lin=2, bias=True),
    dict(bits=4, g=8, act=6),                              # act quant without LET
]


def _flat_params(p):
    keys = []
    for name in ("gamma_logit", "beta_logit", "s", "delta"):
        for i, a in enumerate(p[name]):
            if a is not None:
                keys.append((name, i))
    return keys


@pytest.mark.parametrize("case", FD_CASES, ids=[str(c) for c in FD_CASES])
def test_ste_gradients_match_finite_differences(case):
    case = dict(case)
    bias = case.pop("bias", False)
    rng = np.random.default_rng(11)
    desc = _tiny_desc(T=8, c_in=32, c_out=8, **case)
    X, Y, p = _tiny_params(desc, rng, bias=bias)
    p = {k: [None if a is None else np.asarray(a, np.float64) for a in v] for k, v in p.items()}
    loss, out = block_step(desc, X, Y, p, ft=np.float64)
    frz = freeze(desc, X, Y, p)
    np.testing.assert_allclose(surrogate_loss(desc, X, Y, p, frz), loss, rtol=1e-12)
    grads = {"gamma_logit": out["d_gamma_logit"], "beta_logit": out["d_beta_logit"],
             "s": out["d_s"], "delta": out["d_delta"]}
    for name, i in _flat_params(p):
        base = p[name][i]
        fd = np.zeros(base.size)
        for j in range(base.size):
            eps = 1e-6 * max(1.0, abs(base.flat[j]))
            for sgn in (1, -1):
                q = {k: list(v) for k, v in p.items()}
                arr = base.copy()
                arr.flat[j] += sgn * eps
                q[name][i] = arr
                fd[j] += sgn * surrogate_loss(desc, X, Y, q, frz) / (2 * eps)
        an = np.asarray(grads[name][i]).reshape(-1)
        err = np.max(np.abs(an - fd)) / max(np.max(np.abs(fd)), 1e-30)
        assert err < 1e-6, (name, i, err)
        assert np.max(np.abs(fd)) > 0


def test_fd_detects_a_planted_sign_error():
    """Planting a wrong sign in the shift gradient makes the FD check fail."""
    rng = np.random.default_rng(12)
    desc = _tiny_desc(T=8, c_in=32, c_out=8, bits=4, g=8, let=True, act=4)
    X, Y, p = _tiny_params(desc, rng)
    p = {k: [None if a is None else np.asarray(a, np.float64) for a in v] for k, v in p.items()}
    _, out = block_step(desc, X, Y, p, ft=np.float64)
    frz = freeze(desc, X, Y, p)
    base = p["delta"][0]
    j = 3
    q = {k: list(v) for k, v in p.items()}
    fd = 0.0
    for sgn in (1, -1):
        arr = base.copy()
        arr[j] += sgn * 1e-6
        q["delta"][0] = arr
        fd += sgn * surrogate_loss(desc, X, Y, q, frz) / 2e-6
    assert abs(out["d_delta"][0][j] - fd) < 1e-6 * abs(fd) + 1e-12
    assert abs(-out["d_delta"][0][j] - fd) > 1e-3 * abs(fd)


def test_fp32_spec_and_fp64_agree():
    rng = np.random.default_rng(13)
    desc = _tiny_desc(T=16, c_in=64, c_out=16, bits=4, g=16, let=True, act=8)
    X, Y, p = _tiny_params(desc, rng)
    l32, o32 = block_step(desc, X, Y, p)
    l64, o64 = block_step(desc, X, Y, p, ft=np.float64)
    np.testing.assert_allclose(l32, l64, rtol=1e-3)
    for a, b in zip(o32["d_gamma_logit"], o64["d_gamma_logit"]):
        assert np.max(np.abs(a - b)) / np.max(np.abs(b)) < 2e-2


# ---------------------------------------------------------------- AdamW
def test_adamw_first_step_closed_form():
    """Step 1: m_hat = g, v_hat = g^2, so the update is -lr g / (|g| + eps)."""
    rng = np.random.default_rng(4)
    g = rng.standard_normal(100) * 10.0 ** rng.integers(-9, 2, 100)
    p0 = rng.standard_normal(100)
    p, m, v = adamw(p0, g, np.zeros(100), np.zeros(100), 1, 5e-3)
    np.testing.assert_allclose(p - p0, -5e-3 * g / (np.abs(g) + 1e-8), rtol=1e-9, atol=1e-15)


def test_adamw_matches_library_optimizer():
    rng = np.random.default_rng(5)
    p0 = rng.standard_normal(64)
    t = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([t], lr=1e-2, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0)
    p, m, v = p0.copy(), np.zeros(64), np.zeros(64)
    for step in range(1, 8):
        g = rng.standard_normal(64) * 1e-3
        t.grad = torch.tensor(g)
        opt.step()
        p, m, v = adamw(p, g, m, v, step, 1e-2)
    np.testing.assert_allclose(p, t.detach().numpy(), rtol=1e-12, atol=1e-14)


def test_fp_target_worked_product_with_bias():
    c = GOLD["fp_target_worked"]
    for bf16 in (True, False):
        y = fp_target(np.float32(c["x"]), np.float32(c["w"]), np.float32(c["b"]), bf16=bf16)
        assert y.dtype == np.float32
        np.testing.assert_array_equal(y, np.float32(c["y"]))
    # no bias: the product alone
    y = fp_target(np.float32(c["x"]), np.float32(c["w"]), None)
    np.testing.assert_array_equal(y, np.float32(c["y"]) - np.float32(c["b"])[None, :])


def test_fp_target_rounds_through_fp32_before_bf16():
    """The exact sum lies just above a bf16 midpoint; its fp32 rounding lands
    on the midpoint, which ties to even.  Pins the two-step rounding of the
    target (fp32 accumulator, then bf16 storage)."""
    c = GOLD["fp_target_double_rounding"]
    X, W = np.float32(c["x"]), np.float32(c["w"])
    for b, two, direct in zip(c["b_cases"], c["y_two_step"], c["y_direct"]):
        y = fp_target(X, W, np.float32([b]), bf16=True)
        assert y[0, 0] == np.float32(two), (b, y)
        assert y[0, 0] != np.float32(direct)
        # the fp32 target keeps the fp32 sum (1 + 2^-8 or 1.5 + 2^-8)
        y32 = fp_target(X, W, np.float32([b]), bf16=False)
        assert y32[0, 0] == np.float32(b + 1.0 + 2.0 ** -8)
