"""GPU parity of oq_block_calib_step against the oracle's block step.

Each workload keeps the shape structure of its full-size configuration
(seven LLaMA linears on four sites, GQA k/v, LET on three sites, per-token
activation quantisation, per-channel or grouped weights) at sizes the oracle
finishes in seconds.  Most token counts leave a ragged last tile (the
gradient products then use transposed copies); the multiples of 64 take the
direct path that reads X^, dY^T and W^ as stored.
Bar: loss, row losses and every gradient within 2e-2 normwise relative error
(bf16 matrix-core products); the fp32 workload within 1e-4."""
import numpy as np
import pytest
import torch

from oracle.adamw import LR_LET, LR_LWC, adamw
from oracle.block import block_step
from oracle.quant import lwc_fwd
from paper_2308_13137_amd import configs, oq
from tests.cases import dev, make_problem, normwise, small_llama

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
TOL_F32 = 1e-4

WORKLOADS = [
    configs.C1,
    small_llama("c2_small", hidden=256, ffn=768, T=264, w_bits=3, group=128),
    small_llama("c3_small", hidden=256, ffn=512, T=264, w_bits=4, let=True, act_bits=4),
    small_llama("c4_small", hidden=320, ffn=832, T=136, w_bits=2, group=64),
    small_llama("c5_small", hidden=512, ffn=1024, T=200, w_bits=4, group=128, kv=128, sigma=0.015),
    small_llama("let_noact", hidden=256, ffn=512, T=128, w_bits=4, group=64, let=True),
    # token counts that are multiples of 64: the gradient products read X^, dY^T
    # and W^ as stored instead of transposed copies
    small_llama("c3_t256", hidden=256, ffn=512, T=256, w_bits=4, let=True, act_bits=4),
    small_llama("c2_t320", hidden=256, ffn=768, T=320, w_bits=3, group=128),
    small_llama("c5_t192", hidden=512, ffn=1024, T=192, w_bits=4, group=128, kv=128, sigma=0.015),
    # long token runs over few output tiles: the weight gradient splits its
    # token (K) range into 8 (T=8192) or 4 (T=4096) parts summed afterwards
    small_llama("c2_t8192", hidden=256, ffn=768, T=8192, w_bits=3, group=128),
    small_llama("c3_t4096", hidden=256, ffn=512, T=4096, w_bits=4, let=True, act_bits=4),
    # without LET, unsplit weight gradients with power-of-two groups take the
    # LWC backward in their epilogue: groups of 8 to 256 weights (one lane to
    # four column waves per group), ragged row and column tiles
    small_llama("g64_t256", hidden=320, ffn=832, T=256, w_bits=2, group=64),
    small_llama("g256_t128", hidden=512, ffn=1024, T=128, w_bits=4, group=256),
    small_llama("g32_t192", hidden=256, ffn=512, T=192, w_bits=3, group=32),
    small_llama("g8_t128", hidden=256, ffn=512, T=128, w_bits=2, group=8),
]


def run_gpu(w, P, update=False, blk=None):
    dt = torch.bfloat16 if w.bf16 else torch.float32
    if blk is None:
        blk = oq.Block(w.T, [(s.width, s.let, s.act_bits) for s in w.sites],
                       [(l.site, l.c_out, l.bits, l.group) for l in w.linears], dtype=dt)
    X = [dev(x, dt) for x in P["X"]]
    Y = [dev(np.ascontiguousarray(y.T), dt) for y in P["Y"]]          # channel-major target
    W = [dev(x, dt) for x in P["W"]]
    gl = [dev(x) for x in P["gamma_logit"]]
    bl = [dev(x) for x in P["beta_logit"]]
    s = [None if x is None else dev(x) for x in P["s"]]
    d = [None if x is None else dev(x) for x in P["delta"]]
    B = [None if x is None else dev(x) for x in P["B"]]
    loss = blk.step(X, Y, W, gl, bl, s=s, delta=d, B=B, update=update)
    torch.cuda.synchronize()
    return blk, float(loss.cpu()), gl, bl, s, d


def oracle_step(w, P):
    params = dict(W=P["W"], B=P["B"], gamma_logit=P["gamma_logit"], beta_logit=P["beta_logit"],
                  s=P["s"], delta=P["delta"])
    return block_step(w.oracle_desc(), P["X"], P["Y"], params)


@pytest.mark.parametrize("w", WORKLOADS, ids=[w.name for w in WORKLOADS])
@pytest.mark.parametrize("logit", ["init", "random"])
def test_block_step_parity(w, logit):
    print(f"block step {w.name} T={w.T} logits={logit}", flush=True)
    # biases on a grouped LET workload (let_fold's kernel) and a per-channel
    # one (the bias folded into the whole-row LWC forward)
    P = make_problem(w, seed=3, logit=logit, bias=(w.name in ("let_noact", "c3_t256")))
    blk, loss, *_ = run_gpu(w, P)
    ref_loss, ref = oracle_step(w, P)
    tol = TOL_BF16 if w.bf16 else TOL_F32
    errs = {"loss": abs(loss - ref_loss) / abs(ref_loss)}
    for l in range(len(w.linears)):
        errs[f"dgl{l}"] = normwise(blk.d_gamma[l].cpu().numpy(), ref["d_gamma_logit"][l])
        errs[f"dbl{l}"] = normwise(blk.d_beta[l].cpu().numpy(), ref["d_beta_logit"][l])
        errs[f"row{l}"] = normwise(blk.row_loss[l].cpu().numpy(), ref["row_loss"][l])
    for k, site in enumerate(w.sites):
        if site.let:
            errs[f"ds{k}"] = normwise(blk.d_s[k].cpu().numpy(), ref["d_s"][k])
            errs[f"dd{k}"] = normwise(blk.d_delta[k].cpu().numpy(), ref["d_delta"][k])
    worst = max(errs, key=errs.get)
    print(f"  worst {worst} = {errs[worst]:.3e}", flush=True)
    assert errs[worst] < tol, errs


# 2048-wide sites over 64 tokens: a handful of output tiles and K = 2048, so
# the forward product splits its K range (2 parts, summed by the residual
# pass) and the weight gradient takes the fused LWC backward
FSPLIT = small_llama("fsplit_t64", hidden=2048, ffn=256, T=64, w_bits=4, group=128, kv=256)


def test_block_step_parity_split_forward():
    test_block_step_parity(FSPLIT, "random")


# LET + W4A4 over 65,536 tokens: the input gradient reads a transposed copy
# of W^ (from 65,536 tokens on) and the weight gradients split K in 8
LONG_LET = small_llama("c3_t65536", hidden=128, ffn=256, T=65536, w_bits=4, let=True, act_bits=4)


def test_block_step_parity_long_let():
    test_block_step_parity(LONG_LET, "init")


def test_block_step_is_deterministic():
    w = WORKLOADS[2]
    P = make_problem(w, seed=4)
    blk, l1, *_ = run_gpu(w, P)
    g1 = [t.clone() for t in blk.d_gamma + blk.d_beta] + [blk.d_s[0].clone(), blk.d_delta[0].clone()]
    _, l2, *_ = run_gpu(w, P, blk=blk)
    g2 = blk.d_gamma + blk.d_beta + [blk.d_s[0], blk.d_delta[0]]
    assert l1 == l2
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_twenty_step_trajectory():
    """Twenty AdamW steps on a fixed batch (the 13B-shaped W2A16 g64 workload,
    scaled down): the GPU loss trajectory follows the oracle's."""
    w = small_llama("c4_traj", hidden=256, ffn=512, T=128, w_bits=2, group=64)
    P = make_problem(w, seed=5)
    blk = None
    st = {}
    params = dict(W=P["W"], B=P["B"], gamma_logit=[g.copy() for g in P["gamma_logit"]],
                  beta_logit=[b.copy() for b in P["beta_logit"]], s=P["s"], delta=P["delta"])
    mv = {k: [np.zeros_like(g, np.float64) for g in params[k]] for k in ("gamma_logit", "beta_logit")}
    vv = {k: [np.zeros_like(g, np.float64) for g in params[k]] for k in ("gamma_logit", "beta_logit")}
    dt = torch.bfloat16
    blk = oq.Block(w.T, [(s.width, s.let, s.act_bits) for s in w.sites],
                   [(l.site, l.c_out, l.bits, l.group) for l in w.linears], dtype=dt)
    blk.init_optimizer()
    X = [dev(x, dt) for x in P["X"]]
    Y = [dev(np.ascontiguousarray(y.T), dt) for y in P["Y"]]
    W = [dev(x, dt) for x in P["W"]]
    gl = [dev(x) for x in P["gamma_logit"]]
    bl = [dev(x) for x in P["beta_logit"]]
    ours, refs = [], []
    for step in range(1, 21):
        ours.append(float(blk.step(X, Y, W, gl, bl, update=True).cpu()))
        rl, g = block_step(w.oracle_desc(), P["X"], P["Y"], params)
        refs.append(rl)
        for key, gk in (("gamma_logit", "d_gamma_logit"), ("beta_logit", "d_beta_logit")):
            for l in range(len(w.linears)):
                p, mv[key][l], vv[key][l] = adamw(params[key][l], g[gk][l], mv[key][l],
                                                  vv[key][l], step, LR_LWC)
                params[key][l] = p.astype(np.float32)
    print("  loss gpu", ["%.4e" % x for x in ours[::5]], "oracle", ["%.4e" % x for x in refs[::5]])
    assert refs[-1] < refs[0]
    assert ours[-1] < ours[0]
    for a, b in zip(ours, refs):
        assert abs(a - b) / abs(b) < TOL_BF16
    for l in range(len(w.linears)):
        assert normwise(gl[l].cpu().numpy(), params["gamma_logit"][l]) < 1e-3


def _segments(w, n_seg, seed):
    """One problem of n_seg * T tokens cut into n_seg calibration segments of
    T tokens (rows of X and of the token-major targets); LET is initialised
    over all of them, once per block as Algorithm 1 does."""
    P = make_problem(w.with_tokens(w.T * n_seg), seed=seed)
    segs = []
    for g in range(n_seg):
        rows = slice(g * w.T, (g + 1) * w.T)
        segs.append(dict(X=[x[rows] for x in P["X"]], Y=[y[rows] for y in P["Y"]]))
    return P, segs


def _device_segments(w, segs):
    dt = torch.bfloat16 if w.bf16 else torch.float32
    Xs = [[dev(np.ascontiguousarray(x), dt) for x in sg["X"]] for sg in segs]
    Ys = [[dev(np.ascontiguousarray(y.T), dt) for y in sg["Y"]] for sg in segs]
    return Xs, Ys


def _new_block(w, P):
    dt = torch.bfloat16 if w.bf16 else torch.float32
    blk = oq.Block(w.T, [(s.width, s.let, s.act_bits) for s in w.sites],
                   [(l.site, l.c_out, l.bits, l.group) for l in w.linears], dtype=dt)
    blk.init_optimizer()
    W = [dev(x, dt) for x in P["W"]]
    gl = [dev(x) for x in P["gamma_logit"]]
    bl = [dev(x) for x in P["beta_logit"]]
    s = [None if x is None else dev(x) for x in P["s"]]
    d = [None if x is None else dev(x) for x in P["delta"]]
    return blk, W, gl, bl, s, d


def test_calibrate_loop_equals_step_sequence():
    """oq_block_calibrate (epochs x segments inside the library) gives bit for
    bit what the same steps issued one by one give: losses, logits, s, delta."""
    w = small_llama("c3_loop", hidden=256, ffn=512, T=128, w_bits=4, let=True, act_bits=4)
    P, segs = _segments(w, 3, seed=7)
    Xs, Ys = _device_segments(w, segs)
    a = _new_block(w, P)
    la = a[0].calibrate(Xs, Ys, a[1], a[2], a[3], epochs=2, s=a[4], delta=a[5])
    b = _new_block(w, P)
    lb = []
    for _ in range(2):
        for g in range(3):
            lb.append(float(b[0].step(Xs[g], Ys[g], b[1], b[2], b[3], s=b[4], delta=b[5],
                                      update=True).cpu()))
    torch.cuda.synchronize()
    assert la.cpu().tolist() == lb
    for ta, tb in zip(a[2] + a[3] + [t for t in a[4] + a[5] if t is not None],
                      b[2] + b[3] + [t for t in b[4] + b[5] if t is not None]):
        assert torch.equal(ta, tb)
    assert a[0].step_count == b[0].step_count == 6


def test_calibrate_loop_follows_oracle():
    """Two epochs over three segments (W3A16 g128, LLaMA-shaped, scaled down):
    the step losses and the final clipping logits follow the oracle running
    the same schedule with the same AdamW (Sec. 4.1 settings)."""
    w = small_llama("c2_loop", hidden=256, ffn=768, T=128, w_bits=3, group=128)
    n_seg, epochs = 3, 2
    P, segs = _segments(w, n_seg, seed=11)
    Xs, Ys = _device_segments(w, segs)
    blk, W, gl, bl, s, d = _new_block(w, P)
    ours = blk.calibrate(Xs, Ys, W, gl, bl, epochs=epochs).cpu().tolist()
    params = dict(W=P["W"], B=P["B"], gamma_logit=[g.copy() for g in P["gamma_logit"]],
                  beta_logit=[g.copy() for g in P["beta_logit"]], s=P["s"], delta=P["delta"])
    mv = {k: [np.zeros_like(g, np.float64) for g in params[k]] for k in ("gamma_logit", "beta_logit")}
    vv = {k: [np.zeros_like(g, np.float64) for g in params[k]] for k in ("gamma_logit", "beta_logit")}
    refs, step = [], 0
    for _ in range(epochs):
        for sg in segs:
            step += 1
            rl, g = block_step(w.oracle_desc(), sg["X"], sg["Y"], params)
            refs.append(rl)
            for key, gk in (("gamma_logit", "d_gamma_logit"), ("beta_logit", "d_beta_logit")):
                for l in range(len(w.linears)):
                    p, mv[key][l], vv[key][l] = adamw(params[key][l], g[gk][l], mv[key][l],
                                                      vv[key][l], step, LR_LWC)
                    params[key][l] = p.astype(np.float32)
    print("  loss gpu", ["%.4e" % x for x in ours], "oracle", ["%.4e" % x for x in refs])
    for a, b in zip(ours, refs):
        assert abs(a - b) / abs(b) < TOL_BF16
    for l in range(len(w.linears)):
        assert normwise(gl[l].cpu().numpy(), params["gamma_logit"][l]) < 1e-3
        assert normwise(bl[l].cpu().numpy(), params["beta_logit"][l]) < 1e-3


def test_iterative_schedule_freezes_one_parameter_set():
    """The ablation's iterative training of LWC and LET alternates which set
    learns: a calibrate call with one learning rate at zero leaves that set
    bit for bit unchanged while the other set moves."""
    w = small_llama("c3_iter", hidden=256, ffn=512, T=128, w_bits=4, let=True, act_bits=4)
    P, segs = _segments(w, 2, seed=13)
    Xs, Ys = _device_segments(w, segs)
    blk, W, gl, bl, s, d = _new_block(w, P)
    let0 = [t.clone() for t in s + d if t is not None]
    lwc0 = [t.clone() for t in gl + bl]
    blk.opt_state.lr_let = 0.0                      # LWC phase
    blk.calibrate(Xs, Ys, W, gl, bl, epochs=1, s=s, delta=d)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(let0, [t for t in s + d if t is not None]))
    assert any(not torch.equal(a, b) for a, b in zip(lwc0, gl + bl))
    lwc1 = [t.clone() for t in gl + bl]
    blk.opt_state.lr_let, blk.opt_state.lr_lwc = 1e-2, 0.0   # LET phase
    blk.calibrate(Xs, Ys, W, gl, bl, epochs=1, s=s, delta=d)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(lwc1, gl + bl))
    assert any(not torch.equal(a, b) for a, b in zip(let0, [t for t in s + d if t is not None]))
