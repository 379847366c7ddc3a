"""Pins for the whole-block oracle (oracle/llama_block.py) against things
other than itself: closed forms of RMSNorm, RoPE and SiLU, the library's
scaled-dot-product attention and a torch rebuild of the full-precision block,
the LET equivalences of Eq. 3 and Eq. 5 through the whole block, and central
finite differences of the frozen-choice surrogate for every trained
parameter (clipping logits of all seven linears, s and delta of three sites,
the [Q, K] scale s_a)."""
import math
import struct

import numpy as np
import pytest
import torch

from oracle import llama_block as lb
from oracle.quant import bf16_round


def tiny_desc(act_bits=4, let=True, H=2, Hkv=1, D=16, F=24, S=6, bits=(3, 4, 4, 3, 4, 3, 4),
              act_sym=False, softmax_bits=16):
    return dict(hidden=D, heads=H, kv_heads=Hkv, ffn=F, seq_len=S, norm_eps=1e-6,
                rope_base=10000.0, w_bits=list(bits), w_group=[8, 8, 16, 8, 8, 16, 8],
                act_bits=act_bits, let=let, act_sym=act_sym, softmax_bits=softmax_bits)


def tiny_params(desc, rng, T):
    D, H, Hkv, F = desc["hidden"], desc["heads"], desc["kv_heads"], desc["ffn"]
    d = D // H
    shapes = [(H * d, D), (Hkv * d, D), (Hkv * d, D), (D, H * d), (F, D), (F, D), (D, F)]
    W = [rng.standard_normal(sh) * 0.3 for sh in shapes]
    gl = [rng.uniform(1.0, 4.0, (sh[0], sh[1] // g)) for sh, g in zip(shapes, desc["w_group"])]
    bl = [rng.uniform(1.0, 4.0, a.shape) for a in gl]
    p = dict(W=W, gamma_logit=gl, beta_logit=bl, g1=rng.uniform(0.5, 1.5, D),
             g2=rng.uniform(0.5, 1.5, D),
             s=[rng.uniform(0.5, 2.0, D), rng.uniform(0.5, 2.0, H * d), rng.uniform(0.5, 2.0, D)],
             delta=[rng.standard_normal(D) * 0.2, rng.standard_normal(H * d) * 0.2,
                    rng.standard_normal(D) * 0.2],
             s_a=rng.uniform(0.5, 2.0, Hkv * d))
    h0 = rng.standard_normal((T, D))
    target = lb.fp_block(desc, h0, p) + rng.standard_normal((T, D)) * 0.05
    return h0, target, p


# ---------------------------------------------------------------- smooth pieces
def test_rmsnorm_closed_form():
    y, rstd = lb.rmsnorm(np.array([[3.0, 4.0]]), np.array([1.0, 2.0]), 0.0)
    r = 1.0 / np.sqrt(12.5)
    np.testing.assert_allclose(y[0], [3 * r, 8 * r], rtol=1e-15)
    np.testing.assert_allclose(rstd[0], r, rtol=1e-15)


def test_rmsnorm_backward_is_its_jacobian():
    rng = np.random.default_rng(1)
    h, g, dy = rng.standard_normal((3, 8)), rng.uniform(0.5, 2, 8), rng.standard_normal((3, 8))
    _, rstd = lb.rmsnorm(h, g, 1e-6)
    an = lb.rmsnorm_bwd(h, g, rstd, dy)
    fd = np.zeros_like(h)
    for i in range(3):
        for j in range(8):
            e = np.zeros_like(h)
            e[i, j] = 1e-6
            fd[i, j] = np.sum(dy * (lb.rmsnorm(h + e, g, 1e-6)[0] - lb.rmsnorm(h - e, g, 1e-6)[0])) / 2e-6
    np.testing.assert_allclose(an, fd, rtol=1e-7, atol=1e-9)


def test_rope_closed_forms():
    # d = 2, base irrelevant: the pair (x0, x1) turns by the position angle
    cos, sin = lb.rope_angles(4, 4, 2, 10000.0)
    y = lb.rope(np.tile([[1.0, 0.0]], (4, 1)), 1, 2, cos, sin)
    np.testing.assert_allclose(y, np.stack([np.cos(np.arange(4)), np.sin(np.arange(4))], 1), atol=1e-15)
    rng = np.random.default_rng(2)
    d, S = 8, 7
    cos, sin = lb.rope_angles(2 * S, S, d, 10000.0)
    x = rng.standard_normal((2 * S, 2 * d))
    y = lb.rope(x, 2, d, cos, sin)
    np.testing.assert_allclose(y[0], x[0], atol=0)                  # position 0: identity
    np.testing.assert_allclose(y[S], x[S], atol=0)                  # each sample restarts
    # norms of the pairs (i, i + d/2) are kept; the inverse undoes it
    pr = lambda z: z.reshape(-1, 2, 2, d // 2)
    np.testing.assert_allclose(np.hypot(pr(y)[:, :, 0], pr(y)[:, :, 1]),
                               np.hypot(pr(x)[:, :, 0], pr(x)[:, :, 1]), rtol=1e-13)
    np.testing.assert_allclose(lb.rope(y, 2, d, cos, sin, inverse=True), x, atol=1e-14)
    # <R_m q, R_n k> depends on m - n only
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    cos, sin = lb.rope_angles(S, S, d, 10000.0)
    Rq = lb.rope(np.tile(q, (S, 1)), 1, d, cos, sin)
    Rk = lb.rope(np.tile(k, (S, 1)), 1, d, cos, sin)
    np.testing.assert_allclose(Rq[5] @ Rk[3], Rq[2] @ Rk[0], rtol=1e-12)


def test_silu_closed_form():
    np.testing.assert_allclose(lb.silu(np.array([0.0, 1.0])), [0.0, 1 / (1 + np.exp(-1.0))])
    x = np.linspace(-4, 4, 9)
    fd = (lb.silu(x + 1e-7) - lb.silu(x - 1e-7)) / 2e-7
    np.testing.assert_allclose(lb.silu_grad(x), fd, rtol=1e-7)


@pytest.mark.parametrize("H,Hkv", [(2, 2), (4, 2), (4, 1)])
def test_attention_matches_library_sdpa(H, Hkv):
    rng = np.random.default_rng(3)
    d, S, ns = 8, 7, 2
    q = rng.standard_normal((ns * S, H * d))
    k = rng.standard_normal((ns * S, Hkv * d))
    v = rng.standard_normal((ns * S, Hkv * d))
    out, P, _ = lb.attention(q, k, v, H, Hkv, d, S)
    tq = torch.from_numpy(q).reshape(ns, S, H, d).transpose(1, 2)
    tk = torch.from_numpy(k).reshape(ns, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1)
    tv = torch.from_numpy(v).reshape(ns, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    np.testing.assert_allclose(out, ref.transpose(1, 2).reshape(ns * S, H * d).numpy(), rtol=1e-12,
                               atol=1e-12)
    # the backward against torch's autograd of the same library routine
    do = rng.standard_normal(out.shape)
    dq, dk, dv = lb.attention_bwd(q, k, v, P, do, H, Hkv, d, S)
    tq2 = torch.from_numpy(q).requires_grad_()
    tk2 = torch.from_numpy(k).requires_grad_()
    tv2 = torch.from_numpy(v).requires_grad_()
    o = torch.nn.functional.scaled_dot_product_attention(
        tq2.reshape(ns, S, H, d).transpose(1, 2),
        tk2.reshape(ns, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1),
        tv2.reshape(ns, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1), is_causal=True)
    o.transpose(1, 2).reshape(ns * S, H * d).backward(torch.from_numpy(do))
    for a, b in ((dq, tq2), (dk, tk2), (dv, tv2)):
        np.testing.assert_allclose(a, b.grad.numpy(), rtol=1e-10, atol=1e-12)


def _bf16_py(x):
    """Round-to-nearest-even to bf16 through the float32 bit pattern (struct)."""
    b = struct.unpack("<I", struct.pack("<f", x))[0]
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return struct.unpack("<f", struct.pack("<I", b))[0]


def test_attention_bf16_weights_brute_force():
    """The bf16 reading of the softmax weights, written out per query with
    math/struct on a tiny case: w_j = bf16(2^(t_j - ceil(max t))), out = sum w v
    / sum w (t = q.k log2(e) / sqrt(d), causal)."""
    rng = np.random.default_rng(11)
    H, Hkv, d, S = 2, 1, 4, 5
    q = rng.standard_normal((S, H * d)) * 2
    k = rng.standard_normal((S, Hkv * d))
    v = rng.standard_normal((S, Hkv * d))
    out, _, _ = lb.attention(q, k, v, H, Hkv, d, S, bf16=True)
    for h in range(H):
        for i in range(S):
            t = [sum(q[i, h * d + e] * k[j, e] for e in range(d)) / math.sqrt(d) / math.log(2)
                 for j in range(i + 1)]
            M = math.ceil(max(t))
            w = [_bf16_py(float(np.float32(2.0 ** (tj - M)))) for tj in t]
            for e in range(d):
                ref = sum(w[j] * v[j, e] for j in range(i + 1)) / sum(w)
                assert abs(out[i, h * d + e] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_attention_bf16_weights_properties():
    """A V component shared by every key passes the bf16-weighted mean
    unchanged, and the reading stays within 2^-8 of the exact attention
    relative to the spread of V; P enters dV rounded (within 2^-8)."""
    rng = np.random.default_rng(12)
    H, Hkv, d, S = 2, 2, 8, 16
    q = rng.standard_normal((2 * S, H * d)) * 2
    k = rng.standard_normal((2 * S, Hkv * d))
    u = rng.standard_normal(Hkv * d) * 50
    out_u, _, _ = lb.attention(q, k, np.tile(u, (2 * S, 1)), H, Hkv, d, S, bf16=True)
    np.testing.assert_allclose(out_u, np.tile(u, (2 * S, H // Hkv)), rtol=1e-13)
    v = rng.standard_normal((2 * S, Hkv * d)) + u
    out_b, P, _ = lb.attention(q, k, v, H, Hkv, d, S, bf16=True)
    out_x, _, _ = lb.attention(q, k, v, H, Hkv, d, S)
    spread = np.max(np.abs(v - v.mean(axis=0)))
    assert np.max(np.abs(out_b - out_x)) <= 2.0 ** -8 * spread
    do = rng.standard_normal(out_b.shape)
    _, _, dv_b = lb.attention_bwd(q, k, v, P, do, H, Hkv, d, S, bf16=True)
    _, _, dv_x = lb.attention_bwd(q, k, v, P, do, H, Hkv, d, S)
    Pb = np.abs(P).transpose(0, 1, 3, 2)          # [ns, H, key, query]
    bound = np.zeros_like(dv_x)
    for b in range(2):
        for h in range(H):
            bound[b * S:(b + 1) * S, h * d:(h + 1) * d] = 2.0 ** -8 * Pb[b, h] @ np.abs(
                do[b * S:(b + 1) * S, h * d:(h + 1) * d])
    assert np.all(np.abs(dv_b - dv_x) <= bound + 1e-15)


def test_softmax_quantisation_properties():
    """Q_a on each query row of probabilities: codes in range, within h/2 of
    the row, the causally masked zeros (row minimum 0, so z = 0) stay exactly
    zero, the row's largest probability lands on the top code, and the
    output is the quantised rows times V; at 15 bits the output approaches
    exact attention within 2^-14 of the spread of V."""
    rng = np.random.default_rng(13)
    H, Hkv, d, S = 2, 1, 8, 12
    q = rng.standard_normal((2 * S, H * d)) * 2
    k = rng.standard_normal((2 * S, Hkv * d))
    v = rng.standard_normal((2 * S, Hkv * d))
    rec = {}
    out, P, PH = lb.attention(q, k, v, H, Hkv, d, S, p_bits=4, rec=rec)
    mask = np.triu(np.ones((S, S), bool), 1)
    for b in range(2):
        for h in range(H):
            st = rec[f"pq{b}_{h}"]
            ph, p = PH[b, h], P[b, h]
            assert np.all((st["q"] >= 0) & (st["q"] <= 15))
            hq = st["h"].astype(np.float64)[:, None]
            assert np.all(np.abs(ph - p) <= 0.5 * hq * (1 + 1e-6) + 1e-12)
            assert np.all(ph[:-1][mask[:-1]] == 0.0)
            assert np.all(st["q"][np.arange(S), np.argmax(p, axis=1)] == 15)
            np.testing.assert_allclose(out.reshape(2, S, H, d)[b, :, h, :], ph @ v.reshape(2, S, Hkv, d)[b, :, 0, :],
                                       rtol=1e-12, atol=1e-12)
    out15, _, _ = lb.attention(q, k, v, H, Hkv, d, S, p_bits=15, rec={})
    out_x, _, _ = lb.attention(q, k, v, H, Hkv, d, S)
    assert np.max(np.abs(out15 - out_x)) <= 2.0 ** -14 * np.max(np.abs(v)) * S


def test_fp_block_matches_a_torch_llama_block():
    """The full-precision block against the same block written with torch's
    own ops (RMSNorm by formula, RoPE by complex multiplication, the
    library's causal attention, SiLU)."""
    rng = np.random.default_rng(4)
    desc = tiny_desc(H=4, Hkv=2)
    T = 12
    h0, _, p = tiny_params(desc, rng, T)
    ours = lb.fp_block(desc, h0, p)
    D, H, Hkv, S = 16, 4, 2, 6
    d = D // H
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    h = t(h0)

    def norm(x, g):
        return x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + 1e-6) * t(g)

    pos = torch.arange(T) % S
    freq = 10000.0 ** (-torch.arange(0, d // 2, dtype=torch.float64) * 2 / d)
    rot = torch.polar(torch.ones(T, d // 2, dtype=torch.float64), pos[:, None] * freq[None, :])

    def rope(x, nh):
        x = x.reshape(T, nh, d)
        z = torch.complex(x[..., : d // 2], x[..., d // 2:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], -1)

    W = [t(w) for w in p["W"]]
    x1 = norm(h, p["g1"])
    q = rope(x1 @ W[0].T, H).reshape(T // S, S, H, d).transpose(1, 2)
    k = rope(x1 @ W[1].T, Hkv).reshape(T // S, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1)
    v = (x1 @ W[2].T).reshape(T // S, S, Hkv, d).transpose(1, 2).repeat_interleave(H // Hkv, 1)
    a = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    h1 = h + a.transpose(1, 2).reshape(T, D) @ W[3].T
    x3 = norm(h1, p["g2"])
    ref = h1 + (torch.nn.functional.silu(x3 @ W[4].T) * (x3 @ W[5].T)) @ W[6].T
    np.testing.assert_allclose(ours, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_let_is_an_equivalence_through_the_whole_block():
    """Eq. 3 (s, delta on three sites, folded into the weights and biases) and
    Eq. 5 (s_a on Q and K) change nothing without quantisation: the block's
    loss equals that of the full-precision block for any s, delta, s_a."""
    rng = np.random.default_rng(5)
    desc = dict(tiny_desc(act_bits=16, let=True), w_quant=False)
    T = 12
    h0, target, p = tiny_params(desc, rng, T)
    fp = lb.fp_block(desc, h0, p)
    ref = float(np.mean((fp - target) ** 2))
    loss, c = lb.block_forward(desc, h0, target, p, ft=np.float64)
    np.testing.assert_allclose(loss, ref, rtol=1e-12)
    np.testing.assert_allclose(c["h2"], fp, rtol=1e-11, atol=1e-12)
    # a wrong sign in the [Q, K] scale (s_a on both sides) breaks it
    p2 = dict(p, s_a=p["s_a"] * 1.7)
    loss2, _ = lb.block_forward(desc, h0, target, p2, ft=np.float64)
    np.testing.assert_allclose(loss2, ref, rtol=1e-12)


# ---------------------------------------------------------------- finite differences
FD_CASES = [dict(act_bits=4, let=True), dict(act_bits=16, let=True), dict(act_bits=16, let=False),
            dict(act_bits=3, let=True, H=4, Hkv=2), dict(act_bits=4, let=True, act_sym=True),
            dict(act_bits=4, let=True, softmax_bits=4), dict(act_bits=16, let=True, softmax_bits=6)]


@pytest.mark.parametrize("case", FD_CASES, ids=[str(c) for c in FD_CASES])
def test_block_gradients_match_finite_differences(case):
    rng = np.random.default_rng(6)
    desc = tiny_desc(**case)
    T = 12
    h0, target, p = tiny_params(desc, rng, T)
    loss, g = lb.block_step(desc, h0, target, p, ft=np.float64)
    frz = lb.freeze(desc, h0, target, p)
    np.testing.assert_allclose(lb.surrogate_loss(desc, h0, target, p, frz), loss, rtol=1e-12)
    names = [("gamma_logit", "d_gamma_logit"), ("beta_logit", "d_beta_logit")]
    if desc["let"]:
        names += [("s", "d_s"), ("delta", "d_delta")]
    checks = [(n, gn, i) for n, gn in names for i in range(len(p[n]))]
    if desc["let"]:
        checks.append(("s_a", "d_s_a", None))
    rs = np.random.default_rng(7)
    for name, gname, i in checks:
        base = p[name] if i is None else p[name][i]
        an = np.asarray(g[gname] if i is None else g[gname][i]).reshape(-1)
        idx = rs.choice(base.size, size=min(6, base.size), replace=False)
        for j in idx:
            eps = 1e-6 * max(1.0, abs(base.flat[j]))
            fd = 0.0
            for sgn in (1, -1):
                arr = np.array(base, np.float64, copy=True)
                arr.flat[j] += sgn * eps
                q = dict(p)
                if i is None:
                    q[name] = arr
                else:
                    q[name] = list(p[name])
                    q[name][i] = arr
                fd += sgn * lb.surrogate_loss(desc, h0, target, q, frz) / (2 * eps)
            scale = max(np.max(np.abs(an)), 1e-30)
            # (without activation quantisation s_a cancels exactly: its gradient is 0
            # and the difference quotient is rounding noise of the loss)
            assert abs(an[j] - fd) <= 1e-6 * scale + 1e-9 * max(1.0, loss), (name, i, j, an[j], fd)


def test_fd_detects_a_planted_error_in_the_attention_backward():
    """A 1% error planted in the attention backward's dQ makes the
    finite-difference check of s_a fail (with activation quantisation on, s_a
    carries a gradient)."""
    rng = np.random.default_rng(8)
    desc = tiny_desc(act_bits=4, let=True)
    h0, target, p = tiny_params(desc, rng, 12)
    frz = lb.freeze(desc, h0, target, p)
    j = 3
    fd = 0.0
    for sgn in (1, -1):
        q = dict(p, s_a=p["s_a"].copy())
        q["s_a"][j] += sgn * 1e-6
        fd += sgn * lb.surrogate_loss(desc, h0, target, q, frz) / 2e-6
    _, g_ok = lb.block_step(desc, h0, target, p, ft=np.float64)
    good = lb.attention_bwd
    try:
        def bad(*a, **kw):
            dq, dk, dv = good(*a, **kw)
            return dq * 1.01, dk, dv
        lb.attention_bwd = bad
        _, g_bad = lb.block_step(desc, h0, target, p, ft=np.float64)
    finally:
        lb.attention_bwd = good
    assert abs(g_ok["d_s_a"][j] - fd) <= 1e-6 * abs(fd)
    assert abs(g_bad["d_s_a"][j] - fd) > 1e-4 * abs(fd)


# ---------------------------------------------------------------- Algorithm 1 over a stack
def _stack(desc, rng, n_blocks, T):
    blocks = []
    for _ in range(n_blocks):
        _, _, p = tiny_params(desc, rng, T)
        # the trained tensors are fp32, as the kernels keep them
        for k in ("gamma_logit", "beta_logit", "s", "delta"):
            p[k] = [np.asarray(a, np.float32) for a in p[k]]
        p["s_a"] = np.asarray(p["s_a"], np.float32)
        blocks.append(p)
    return blocks


def test_algorithm1_without_learning_composes_the_blocks():
    """With both learning rates 0 nothing moves: every loss of block i is
    one step's loss at its initial parameters, against targets that are the
    full-precision blocks composed (each output rounded to bf16), from the
    quantised blocks composed at their initial parameters."""
    desc = tiny_desc()
    rng = np.random.default_rng(41)
    S = desc["seq_len"]
    blocks = _stack(desc, rng, 2, S)
    samples = [rng.standard_normal((S, desc["hidden"])) for _ in range(2)]
    losses, trained, xq = lb.algorithm1(desc, blocks, samples, epochs=2, lr_lwc=0.0, lr_let=0.0)
    fp1 = [bf16_round(lb.fp_block(desc, x, blocks[0])) for x in samples]
    fp2 = [bf16_round(lb.fp_block(desc, x, blocks[1])) for x in fp1]
    q1 = [bf16_round(lb.block_forward(desc, x, t, blocks[0])[1]["h2"]) for x, t in zip(samples, fp1)]
    want0 = [lb.block_step(desc, x, t, blocks[0])[0] for x, t in zip(samples, fp1)]
    want1 = [lb.block_step(desc, x, t, blocks[1])[0] for x, t in zip(q1, fp2)]
    np.testing.assert_allclose(losses[0], want0 * 2, rtol=1e-12)
    np.testing.assert_allclose(losses[1], want1 * 2, rtol=1e-12)
    q2 = [bf16_round(lb.block_forward(desc, x, t, blocks[1])[1]["h2"]) for x, t in zip(q1, fp2)]
    for a, b in zip(xq, q2):
        np.testing.assert_array_equal(a, b)
    for P, P0 in zip(trained, blocks):
        for a, b in zip(P["gamma_logit"], P0["gamma_logit"]):
            np.testing.assert_allclose(a, b, rtol=1e-7)


def test_algorithm1_first_step_of_every_block_is_a_fresh_adam_step():
    """Each block gets a fresh AdamW state: its first update moves every
    parameter with a nonzero gradient by its learning rate (Adam's first
    bias-corrected step is lr g / (|g| + eps)), the clipping logits by 5e-3
    and s, delta, s_a by 1e-2, in the second block as in the first."""
    desc = tiny_desc()
    rng = np.random.default_rng(42)
    S = desc["seq_len"]
    blocks = _stack(desc, rng, 2, S)
    samples = [rng.standard_normal((S, desc["hidden"]))]
    _, trained, _ = lb.algorithm1(desc, blocks, samples, epochs=1)
    def check(moved, lr, key):
        # no element moves further than lr (up to the fp32 storage of p);
        # the typical one (|g| >> eps) moves lr
        assert np.max(moved) <= lr * (1 + 1e-4) + 1e-6, key
        assert abs(np.median(moved) / lr - 1) < 2e-3, (key, np.median(moved))
    for P, P0 in zip(trained, blocks):
        for key, lr in (("gamma_logit", 5e-3), ("beta_logit", 5e-3), ("s", 1e-2), ("delta", 1e-2)):
            moved = np.concatenate([np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float32)).ravel()
                                    for a, b in zip(P[key], P0[key])])
            check(moved, lr, key)
        check(np.abs(np.asarray(P["s_a"], np.float64) - np.asarray(P0["s_a"], np.float32)), 1e-2, "s_a")


def test_algorithm1_training_lowers_the_loss():
    """Twenty epochs over two samples lower every block's loss."""
    desc = tiny_desc(act_bits=16)
    rng = np.random.default_rng(43)
    S = desc["seq_len"]
    blocks = _stack(desc, rng, 2, S)
    samples = [rng.standard_normal((S, desc["hidden"])) for _ in range(2)]
    losses, _, _ = lb.algorithm1(desc, blocks, samples, epochs=20)
    for bl_ in losses:
        assert sum(bl_[-2:]) < 0.9 * sum(bl_[:2]), bl_
