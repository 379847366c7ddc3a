"""Pins for the oracle's quantiser variants (the appendix's comparison of LWC
with PACT and LSQ run inside the same pipeline, and symmetric absmax
activation quantisation): hand-worked examples, reductions to the MinMax
quantiser the other pins fix, and central finite differences of each
variant's straight-through surrogate through a whole block step."""
import numpy as np
import pytest

from oracle.block import block_step
from oracle.quant import (act_fwd, act_sym_bwd, act_sym_fwd, lsq_bwd, lsq_fwd, lsq_grad_scale,
                          lwc_fwd, pact_bwd, pact_fwd, wquant_init)
from oracle.surrogate import freeze, surrogate_loss


# ---------------------------------------------------------------- worked examples
def test_pact_worked_example():
    """bits 2, w = [-1, -0.5, 0, 0.5, 1.5]:
    hi = 1, lo = -1: h = 2/3, 1/h -> 1.5, z = -round(-1.5) = 2; w/h rounded
    [-2, -1, 0, 1, 2] + 2 = [0, 1, 2, 3, 4]: only the last code saturates
    (above), so with g = [1..5]: dhi = 5, dlo = 0, dw = [1, 2, 3, 4, 0].
    lo = -0.5: h = 0.5, z = 1, codes before the clamp [-1, 0, 1, 2, 4]: the
    first saturates below, the last above: dhi = 5, dlo = 1, dw = [0, 2, 3, 4, 0]."""
    W = np.float32([[-1.0, -0.5, 0.0, 0.5, 1.5]])
    g = np.float32([[1, 2, 3, 4, 5]])
    st = pact_fwd(W, np.float32([[1.0]]), np.float32([[-1.0]]), 2, 5)
    assert st["codes"][0].tolist() == [0, 1, 2, 3, 3] and st["z"][0] == 2
    r = pact_bwd(st, g)
    assert r["d_p1"][0, 0] == 5 and r["d_p2"][0, 0] == 0
    assert r["dW_tilde"][0].tolist() == [1, 2, 3, 4, 0]
    st = pact_fwd(W, np.float32([[1.0]]), np.float32([[-0.5]]), 2, 5)
    assert st["c"][0].tolist() == [-1, 0, 1, 2, 4] and st["h"][0] == 0.5
    r = pact_bwd(st, g)
    assert r["d_p1"][0, 0] == 5 and r["d_p2"][0, 0] == 1
    assert r["dW_tilde"][0].tolist() == [0, 2, 3, 4, 0]


def test_lsq_worked_example():
    """bits 2, group 4, h = 0.5, z = 1.4 (rounded to 1), w = [-0.5, 0, 0.6, 2]:
    w/h = [-1, 0, 1.2, 4] -> round + 1 = [0, 1, 2, 5] -> clamp [0, 1, 2, 3];
    q - z = [-1, 0, 1, 2].  With g = 1: S_h = 0 + 0 - 0.2 + 2 = 1.8, S_z = 1;
    gradient scale 1/sqrt(4 * 3): dh = 1.8/sqrt(12), dz = -0.5/sqrt(12)."""
    W = np.float32([[-0.5, 0.0, 0.6, 2.0]])
    st = lsq_fwd(W, np.float32([[0.5]]), np.float32([[1.4]]), 2, 4)
    assert st["codes"][0].tolist() == [0, 1, 2, 3] and st["z"][0] == 1
    np.testing.assert_array_equal(st["W_dq"][0], np.float32([-0.5, 0.0, 0.5, 1.0]))
    assert lsq_grad_scale(4, 2) == 1.0 / np.sqrt(12.0)
    r = lsq_bwd(st, np.ones((1, 4)))
    np.testing.assert_allclose(r["d_p1"][0, 0], 1.8 / np.sqrt(12.0), rtol=1e-6)
    np.testing.assert_allclose(r["d_p2"][0, 0], -0.5 / np.sqrt(12.0), rtol=1e-12)
    assert r["dW_tilde"][0].tolist() == [1, 1, 1, 0]


def test_symmetric_activation_worked_example():
    """bits 4 (7 steps each side, zero point 8), x = [-3.5, 1, 0.25, 3.5]:
    |x| peaks at indices 0 and 3, the lowest (0, sign -1) carries it;
    h = 3.5/7 = 0.5, x/h = [-7, 2, 0.5, 7] -> round half to even [-7, 2, 0, 7]
    + 8 = [1, 10, 8, 15].  With g = 1: dh = sum((q - z) - x/h) = -0.5,
    d|x|max = -0.5/7, so dx = [1 + 1/14, 1, 1, 1]."""
    st = act_sym_fwd(np.float32([[-3.5, 1.0, 0.25, 3.5]]), 4)
    assert st["codes"][0].tolist() == [1, 10, 8, 15]
    assert st["h"][0] == 0.5 and st["z"][0] == 8 and st["i_ab"][0] == 0
    np.testing.assert_array_equal(st["X_dq"][0], np.float32([-3.5, 1.0, 0.0, 3.5]))
    dx = act_sym_bwd(st, np.ones((1, 4)))
    np.testing.assert_allclose(dx[0], [1 + 1 / 14, 1, 1, 1], rtol=1e-12)


# ---------------------------------------------------------------- reductions to MinMax
@pytest.mark.parametrize("bits,group", [(2, 64), (3, 128), (4, 32), (8, 256)])
def test_minmax_initialised_variants_equal_unit_clip_lwc(bits, group):
    """At their MinMax initialisation PACT (hi, lo = max, min) and LSQ (h, z of
    MinMax) quantise exactly as LWC at clip strength 1 (sigmoid(30) = 1.0f),
    which the textbook-RTN pin fixes."""
    rng = np.random.default_rng(bits * 100 + group)
    W = (rng.standard_normal((24, 512)) * 0.02).astype(np.float32)
    ref = lwc_fwd(W, np.full((24, 512 // group), 30.0), np.full((24, 512 // group), 30.0), bits, group)
    hi, lo = wquant_init(W, bits, group, "pact")
    np.testing.assert_array_equal(hi, W.reshape(-1, group).max(axis=1).reshape(hi.shape))
    st = pact_fwd(W, hi, lo, bits, group)
    assert np.array_equal(st["codes"], ref["codes"]) and np.array_equal(st["W_dq"], ref["W_dq"])
    h, z = wquant_init(W, bits, group, "lsq")
    st = lsq_fwd(W, h, z, bits, group)
    assert np.array_equal(st["codes"], ref["codes"]) and np.array_equal(st["W_dq"], ref["W_dq"])


def test_symmetric_activation_invariants():
    rng = np.random.default_rng(3)
    X = (rng.standard_normal((64, 256)) * rng.uniform(0.1, 5, (64, 1))).astype(np.float32)
    for bits in (3, 4, 8):
        st = act_sym_fwd(X, bits)
        qs = 2 ** (bits - 1) - 1
        off = st["q"] - st["z"][:, None]
        assert np.all(np.abs(off) <= qs)                       # symmetric range
        assert np.all(st["z"] == 2 ** (bits - 1))
        err = np.abs(st["X_dq"].astype(np.float64) - X)
        assert np.all(err <= st["h"][:, None] * (0.5 + 1e-6))  # nearest grid point
        # the absmax element is represented exactly (its code is +-qs)
        rows = np.arange(64)
        assert np.all(np.abs(off[rows, st["i_ab"]]) == qs)
    # asymmetric MinMax of a row symmetric about 0 uses the same step
    row = np.float32([[-2.0, -1.0, 0.5, 2.0]])
    assert act_sym_fwd(row, 8)["h"][0] == np.float32(2.0) / np.float32(127)
    assert act_fwd(row, 8)["h"][0] == np.float32(4.0) / np.float32(255)


# ---------------------------------------------------------------- finite differences
def _desc(quant, let=False, act=16, act_sym=False, T=8, c_in=32, c_out=8, g=8, bits=3):
    return dict(T=T, bf16=False, sites=[dict(width=c_in, let=let, act_bits=act, act_sym=act_sym)],
                linears=[dict(site=0, c_out=c_out, bits=bits, group=g, quant=quant),
                         dict(site=0, c_out=c_out, bits=bits + 1, group=g * 2, quant=quant)])


def _params(desc, rng):
    T = desc["T"]
    C = desc["sites"][0]["width"]
    X = [rng.standard_normal((T, C))]
    W, gl, bl, Y = [], [], [], []
    for lin in desc["linears"]:
        w = rng.standard_normal((lin["c_out"], C)) * 0.5
        W.append(w)
        s = None
        p1, p2 = wquant_init(w.astype(np.float32), lin["bits"], lin["group"], lin["quant"])
        if lin["quant"] == "pact":                 # thresholds inside the range: both clamp sides active
            p1, p2 = p1 * 0.8, p2 * 0.7
        elif lin["quant"] == "lsq":
            p1, p2 = p1 * 0.7, p2 + 0.3               # a finer step: codes saturate too
        gl.append(np.asarray(p1, np.float64))
        bl.append(np.asarray(p2, np.float64))
        Y.append(X[0] @ w.T + rng.standard_normal((T, lin["c_out"])) * 0.05)
    site = desc["sites"][0]
    s = [rng.uniform(0.5, 2.0, C)] if site["let"] else [None]
    d = [rng.standard_normal(C) * 0.3] if site["let"] else [None]
    return X, Y, dict(W=W, B=[None, None], gamma_logit=gl, beta_logit=bl, s=s, delta=d)


VARIANT_CASES = [dict(quant="pact"), dict(quant="lsq"), dict(quant="pact", let=True),
                 dict(quant="lsq", let=True, act=4), dict(quant="lwc", let=True, act=4, act_sym=True),
                 dict(quant="lsq", let=True, act=3, act_sym=True)]


@pytest.mark.parametrize("case", VARIANT_CASES, ids=[str(c) for c in VARIANT_CASES])
def test_variant_gradients_match_finite_differences(case):
    rng = np.random.default_rng(21)
    desc = _desc(**case)
    X, Y, p = _params(desc, rng)
    loss, out = block_step(desc, X, Y, p, ft=np.float64)
    frz = freeze(desc, X, Y, p)
    np.testing.assert_allclose(surrogate_loss(desc, X, Y, p, frz), loss, rtol=1e-12)
    grads = {"gamma_logit": out["d_gamma_logit"], "beta_logit": out["d_beta_logit"],
             "s": out["d_s"], "delta": out["d_delta"]}
    for name in ("gamma_logit", "beta_logit", "s", "delta"):
        for i, base in enumerate(p[name]):
            if base is None:
                continue
            scale = 1.0
            lin = desc["linears"][i] if name in ("gamma_logit", "beta_logit") else None
            if lin is not None and lin["quant"] == "lsq":
                scale = lsq_grad_scale(lin["group"], lin["bits"])   # LSQ's gradient scale
            fd = np.zeros(base.size)
            for j in range(base.size):
                eps = 1e-6 * max(1.0, abs(base.flat[j]))
                for sgn in (1, -1):
                    q = {k: list(v) for k, v in p.items()}
                    arr = base.copy()
                    arr.flat[j] += sgn * eps
                    q[name][i] = arr
                    fd[j] += sgn * surrogate_loss(desc, X, Y, q, frz) / (2 * eps)
            an = np.asarray(grads[name][i]).reshape(-1) / scale
            err = np.max(np.abs(an - fd)) / max(np.max(np.abs(fd)), 1e-30)
            assert err < 1e-6, (name, i, err)
            assert np.max(np.abs(fd)) > 0, (name, i)


def test_pact_rule_differs_from_the_full_straight_through_gradient():
    """PACT's rule (identity on the clipped weight) is not Eq. 2's full
    straight-through gradient: the same thresholds as LWC bounds give other
    threshold gradients, so the two quantisers are told apart."""
    rng = np.random.default_rng(5)
    W = (rng.standard_normal((4, 64)) * 0.02).astype(np.float32)
    hi, lo = wquant_init(W, 3, 64, "pact")
    g = rng.standard_normal((4, 64))
    r = pact_bwd(pact_fwd(W, hi * 0.8, lo * 0.8, 3, 64), g)
    # LWC at gamma = beta = 0.8 has the same grid (a = 0.8 max, b = 0.8 min)
    from oracle.quant import lwc_bwd
    logit = np.log(0.8 / 0.2)
    st = lwc_fwd(W, np.full((4, 1), logit), np.full((4, 1), logit), 3, 64)
    rl = lwc_bwd(st, g)
    assert not np.allclose(rl["dW_tilde"], r["dW_tilde"])       # LWC routes max/min gradients
