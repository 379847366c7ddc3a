"""GPU parity of each C-ABI entry point against the oracle, on seeded inputs.

Bars: integer codes (and the fp32 h, z that decide them) bit-exact; fp32
elementwise outputs within 1e-5 normwise relative error; matrix products with
fp32 accumulation within 1e-4 (the fp32 accumulation error over K <= 4096
terms, far inside the 2e-2 bar for bf16 GEMM outputs)."""
import numpy as np
import pytest
import torch

from oracle.adamw import adamw as adamw_ref
from oracle.block import fp_target as fp_target_ref
from oracle.let import let_bias, let_init as let_init_ref, let_w, let_x
from oracle.quant import act_bwd, act_fwd, bf16_round, lwc_bwd, lwc_fwd
from paper_2308_13137_amd import inputs, oq
from tests.cases import U32, bf16_exact, dev, normwise, quant_grad_bounds, within

pytestmark = pytest.mark.gpu

TOL_FP32 = 1e-5
TOL_GEMM = 1e-4


def host(t):
    return t.detach().float().cpu().numpy()


# ---------------------------------------------------------------- matrix products
@pytest.mark.parametrize("M,N,K", [(256, 256, 64), (300, 520, 136), (8, 8, 8), (1024, 768, 512),
                                   (257, 1000, 4096), (64, 4096, 8)])
def test_matmul_nt_bf16(M, N, K):
    print(f"matmul bf16 M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 7 + N + K)
    A = bf16_exact(rng.standard_normal((M, K)))
    B = bf16_exact(rng.standard_normal((N, K)))
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    got = host(oq.matmul_nt(dev(A, torch.bfloat16), dev(B, torch.bfloat16)))
    assert normwise(got, ref) < TOL_GEMM
    # bf16 x bf16 products are exact in fp32: only the K-term fp32 sum rounds
    within(got, ref, (K + 2) * U32 * (np.abs(A).astype(np.float64) @ np.abs(B).T.astype(np.float64)),
           "C")
    got16 = host(oq.matmul_nt(dev(A, torch.bfloat16), dev(B, torch.bfloat16), torch.bfloat16))
    assert np.max(np.abs(got16 - ref) / (np.abs(ref) + 1e-3 * np.max(np.abs(ref)))) < 2 ** -7


@pytest.mark.parametrize("a_mn,b_mn", [(False, True), (True, True), (True, False), (False, False)])
@pytest.mark.parametrize("M,N,K", [(256, 256, 64), (392, 1000, 640), (8, 264, 128),
                                   (1024, 768, 4096), (520, 16, 192)])
def test_matmul_operand_layouts(M, N, K, a_mn, b_mn):
    """Operands stored MN-major ([K, M] / [K, N]) are read as stored (the
    step's gradient products); M, N that are not tile multiples exercise the
    clamped tile edges."""
    print(f"matmul layouts a_mn={a_mn} b_mn={b_mn} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 3 + N * 5 + K + 2 * a_mn + b_mn)
    A = bf16_exact(rng.standard_normal((M, K)))
    B = bf16_exact(rng.standard_normal((N, K)))
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    Ad = dev(np.ascontiguousarray(A.T) if a_mn else A, torch.bfloat16)
    Bd = dev(np.ascontiguousarray(B.T) if b_mn else B, torch.bfloat16)
    got = host(oq.matmul(Ad, Bd, a_mn=a_mn, b_mn=b_mn))
    assert normwise(got, ref) < TOL_GEMM
    within(got, ref, (K + 2) * U32 * (np.abs(A).astype(np.float64) @ np.abs(B).T.astype(np.float64)),
           "C")


def test_matmul_operand_layout_unsupported():
    A = torch.zeros((96, 64), dtype=torch.bfloat16, device="cuda")     # K = 96: not a multiple of 64
    B = torch.zeros((96, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(oq.OQError, match="UNSUPPORTED|MN-major"):
        oq.matmul(A, B, a_mn=True, b_mn=True)


@pytest.mark.parametrize("M,N,K", [(64, 64, 16), (130, 70, 264), (256, 256, 256)])
def test_matmul_nt_f32(M, N, K):
    print(f"matmul f32 M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + N + K)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K)).astype(np.float32)
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    got = host(oq.matmul_nt(dev(A), dev(B)))
    assert normwise(got, ref) < TOL_GEMM


@pytest.mark.parametrize("bf16", [True, False])
def test_fp_target(bf16):
    rng = inputs.rng_for(5, int(bf16))
    T, c_in, c_out = 384, 512, 320
    X = inputs.activations(rng, T, c_in)
    W = inputs.weights(rng, c_out, c_in, 0.02, 0.001)
    B = rng.standard_normal(c_out).astype(np.float32) * 0.1
    dt = torch.bfloat16 if bf16 else torch.float32
    if bf16:
        X, W = bf16_exact(X), bf16_exact(W)
    ref = fp_target_ref(X, W, B, bf16=bf16)                  # [T, c_out]
    got = host(oq.fp_target(dev(X, dt), dev(W, dt), dev(B)))  # [c_out, T]
    if bf16:
        # one bf16 rounding of an fp32 sum vs of an fp64 sum: nearly all equal,
        # the rest one bf16 step apart (relative to the output's scale)
        assert np.mean(got == ref.T) > 0.98
        assert normwise(got, ref.T) <= 2.0 ** -8
    else:
        assert normwise(got, ref.T) < TOL_GEMM
    # per element: the fp32 accumulator's error bound, then (bf16 target) at
    # most one bf16 step more than the oracle's single rounding
    acc = (np.abs(X).astype(np.float64) @ np.abs(W).T.astype(np.float64) + np.abs(B)[None, :]).T
    bound = (c_in + 3) * U32 * acc
    if bf16:
        # two roundings to bf16 of values that close can land one bf16 step
        # (at most 2^-7 relative) apart
        bound = bound * (1 + 2.0 ** -7) + 2.0 ** -7 * np.abs(ref.T)
    within(got, ref.T, bound, "Y_fp")


# ---------------------------------------------------------------- LWC
LWC_CASES = [
    dict(c_out=96, c_in=1024, group=128, bits=3, bf16=True),
    dict(c_out=37, c_in=4096, group=4096, bits=4, bf16=True),       # per output channel
    dict(c_out=64, c_in=1000, group=1000, bits=4, bf16=True),       # per channel, ragged row
    dict(c_out=256, c_in=256, group=64, bits=4, bf16=False),        # fp32 linear
    dict(c_out=40, c_in=11008, group=128, bits=2, bf16=True),
    dict(c_out=24, c_in=512, group=32, bits=8, bf16=True),
    dict(c_out=16, c_in=2048, group=512, bits=3, bf16=True),
    dict(c_out=12, c_in=4096, group=128, bits=4, bf16=True, let=True),
    dict(c_out=20, c_in=11008, group=11008, bits=4, bf16=True, let=True),
    # the smallest and the remaining power-of-two groups, with a chunk count
    # that leaves a partial wave step (13 x 17, 7 x 26, 9 x 96 chunks of 8)
    dict(c_out=13, c_in=136, group=8, bits=2, bf16=True),
    dict(c_out=7, c_in=208, group=16, bits=5, bf16=True),
    dict(c_out=9, c_in=768, group=256, bits=6, bf16=False),
    # whole-row groups on the wave-per-row kernels: fp32 rows with s, and
    # two-chunk rows over more rows than one workgroup's waves
    dict(c_out=33, c_in=2048, group=2048, bits=5, bf16=False, let=True),
    dict(c_out=70, c_in=136, group=136, bits=3, bf16=True),
]


def _lwc_inputs(case, seed=0):
    rng = inputs.rng_for(11, seed, case["c_in"], case["group"], case["bits"])
    W = inputs.weights(rng, case["c_out"], case["c_in"], 0.02, 0.001)
    if case["bf16"]:
        W = bf16_exact(W)
    ng = case["c_in"] // case["group"]
    gl = rng.uniform(-1.0, 6.0, (case["c_out"], ng)).astype(np.float32)
    bl = rng.uniform(-1.0, 6.0, (case["c_out"], ng)).astype(np.float32)
    s = rng.uniform(0.3, 3.0, case["c_in"]).astype(np.float32) if case.get("let") else None
    return W, gl, bl, s


@pytest.mark.parametrize("case", LWC_CASES, ids=[str(c) for c in LWC_CASES])
def test_lwc_fwd_codes_bit_exact(case):
    print(f"lwc_fwd {case}", flush=True)
    W, gl, bl, s = _lwc_inputs(case)
    dt = torch.bfloat16 if case["bf16"] else torch.float32
    ref = lwc_fwd(W, gl, bl, case["bits"], case["group"], s=s)
    Wdq, codes, h, z = oq.lwc_fakequant_fwd(dev(W, dt), dev(gl), dev(bl), case["bits"],
                                           case["group"], s=None if s is None else dev(s),
                                           dq_dtype=torch.float32)
    assert np.array_equal(host(h), ref["h_g"])
    assert np.array_equal(host(z), ref["z_g"])
    assert np.array_equal(codes.cpu().numpy(), ref["codes"])
    assert np.array_equal(host(Wdq), ref["W_dq"])
    Wdq16, _, _, _ = oq.lwc_fakequant_fwd(dev(W, dt), dev(gl), dev(bl), case["bits"], case["group"],
                                         s=None if s is None else dev(s), dq_dtype=torch.bfloat16,
                                         codes=False, hz=False)
    assert np.array_equal(host(Wdq16), bf16_round(ref["W_dq"]))


@pytest.mark.parametrize("case", LWC_CASES, ids=[str(c) for c in LWC_CASES])
def test_lwc_bwd(case):
    print(f"lwc_bwd {case}", flush=True)
    W, gl, bl, s = _lwc_inputs(case, seed=1)
    dt = torch.bfloat16 if case["bf16"] else torch.float32
    rng = np.random.default_rng(case["c_in"] + case["c_out"])
    G = rng.standard_normal((case["c_out"], case["c_in"])).astype(np.float32)
    st = lwc_fwd(W, gl, bl, case["bits"], case["group"], s=s)
    ref = lwc_bwd(st, G, W=W, with_s=True)
    dg, db, ds, dwt = oq.lwc_fakequant_bwd(dev(W, dt), dev(gl), dev(bl), case["bits"], case["group"],
                                           dev(G), s=None if s is None else dev(s), want_d_s=True,
                                           want_dW_tilde=True)
    assert normwise(host(dg), ref["d_gamma_logit"]) < TOL_FP32
    assert normwise(host(db), ref["d_beta_logit"]) < TOL_FP32
    assert normwise(host(dwt), ref["dW_tilde"]) < TOL_FP32
    assert normwise(host(ds), ref["d_s"]) < TOL_FP32
    # per element, within the bound the fp32 arithmetic allows
    bx, bg, bb = quant_grad_bounds(st, G)
    within(host(dwt), ref["dW_tilde"], bx.reshape(G.shape), "dW~")
    within(host(dg), ref["d_gamma_logit"], bg.reshape(dg.shape), "d_gamma_logit")
    within(host(db), ref["d_beta_logit"], bb.reshape(db.shape), "d_beta_logit")


# ---------------------------------------------------------------- activations
ACT_CASES = [
    dict(T=96, C=4096, bits=4, let=False), dict(T=77, C=4096, bits=4, let=True),
    dict(T=40, C=11008, bits=4, let=True), dict(T=64, C=1000, bits=8, let=True),
    dict(T=50, C=256, bits=6, let=False, bf16=False), dict(T=33, C=2048, bits=16, let=True),
    # several rows per workgroup (T > 2048), so the backward's row pipeline
    # runs; a ragged 257-chunk row and a plain 4096-channel one
    dict(T=4100, C=2056, bits=4, let=True), dict(T=3000, C=4096, bits=3, let=False),
    # rows wider than 8,192 channels: the backward runs 512 threads per row
    dict(T=1600, C=11008, bits=4, let=False, bf16=False), dict(T=12, C=20480, bits=6, let=True),
]


def _act_inputs(case):
    rng = inputs.rng_for(12, case["T"], case["C"], case["bits"])
    X = inputs.activations(rng, case["T"], case["C"])
    if case.get("bf16", True):
        X = bf16_exact(X)
    s = d = None
    if case["let"]:
        s = rng.uniform(0.3, 3.0, case["C"]).astype(np.float32)
        d = (rng.standard_normal(case["C"]) * 0.2).astype(np.float32)
    return X, s, d


@pytest.mark.parametrize("case", ACT_CASES, ids=[str(c) for c in ACT_CASES])
def test_act_fwd_codes_bit_exact(case):
    print(f"act_fwd {case}", flush=True)
    X, s, d = _act_inputs(case)
    dt = torch.bfloat16 if case.get("bf16", True) else torch.float32
    xt = let_x(X, s, d) if case["let"] else X
    Xq, codes, h, z = oq.act_fakequant_fwd(dev(X, dt), case["bits"], s=None if s is None else dev(s),
                                          delta=None if d is None else dev(d),
                                          dq_dtype=torch.float32)
    if case["bits"] == 16:
        assert np.array_equal(host(Xq), xt)
        return
    ref = act_fwd(xt, case["bits"])
    assert np.array_equal(codes.cpu().numpy(), ref["codes"])
    assert np.array_equal(host(h), ref["h"])
    assert np.array_equal(host(z), ref["z"])
    assert np.array_equal(host(Xq), ref["X_dq"])


@pytest.mark.parametrize("case", ACT_CASES, ids=[str(c) for c in ACT_CASES])
def test_act_bwd(case):
    print(f"act_bwd {case}", flush=True)
    X, s, d = _act_inputs(case)
    dt = torch.bfloat16 if case.get("bf16", True) else torch.float32
    rng = np.random.default_rng(case["T"])
    G = rng.standard_normal(X.shape).astype(np.float32)
    xt = let_x(X, s, d) if case["let"] else X
    bx = None
    if case["bits"] < 16:
        st = act_fwd(xt, case["bits"])
        dxt = act_bwd(st, G)
        bx, _, _ = quant_grad_bounds(st, G)
    else:
        dxt = G.astype(np.float64)
    sv = np.ones(X.shape[1]) if s is None else s.astype(np.float64)
    ref_ds = -np.sum(dxt * xt, axis=0) / sv
    ref_dd = -np.sum(dxt, axis=0) / sv
    gx, ds, dd = oq.act_fakequant_bwd(dev(X, dt), case["bits"], dev(G),
                                      s=None if s is None else dev(s),
                                      delta=None if d is None else dev(d))
    assert normwise(host(gx), dxt) < TOL_FP32
    if bx is not None:
        within(host(gx), dxt, bx, "dX~")
    else:
        assert np.array_equal(host(gx), G)
    assert normwise(host(ds), ref_ds) < TOL_FP32
    assert normwise(host(dd), ref_dd) < TOL_FP32


# ---------------------------------------------------------------- LET, AdamW
@pytest.mark.parametrize("bf16", [True, False])
def test_let_fold(bf16):
    rng = inputs.rng_for(13, int(bf16))
    W = inputs.weights(rng, 72, 1024, 0.02, 0.001)
    W = bf16_exact(W) if bf16 else W
    B = rng.standard_normal(72).astype(np.float32)
    s = rng.uniform(0.3, 3.0, 1024).astype(np.float32)
    d = rng.standard_normal(1024).astype(np.float32)
    dt = torch.bfloat16 if bf16 else torch.float32
    Wt, Bt = oq.let_fold(dev(W, dt), dev(B), dev(s), dev(d), wt_dtype=torch.float32)
    assert np.array_equal(host(Wt), let_w(W, s))
    assert normwise(host(Bt), let_bias(W, B, d)) < TOL_FP32


def test_let_init():
    rng = inputs.rng_for(14)
    X = bf16_exact(inputs.activations(rng, 1000, 512))
    Ws = [bf16_exact(inputs.weights(rng, co, 512, 0.02, 0.001)) for co in (512, 128, 128)]
    s, d = oq.let_init(dev(X, torch.bfloat16), [dev(W, torch.bfloat16) for W in Ws])
    rs, rd = let_init_ref(X, Ws)
    assert np.array_equal(host(s), rs)
    assert normwise(host(d), rd) < TOL_FP32


def test_adamw():
    rng = np.random.default_rng(15)
    n = 10000
    p0 = rng.standard_normal(n).astype(np.float32)
    m0 = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v0 = (rng.uniform(0, 1e-6, n)).astype(np.float32)
    g = (rng.standard_normal(n) * 10.0 ** rng.integers(-9, 0, n)).astype(np.float32)
    p, m, v = dev(p0), dev(m0), dev(v0)
    oq.adamw_step(p, dev(g), m, v, step=3, lr=5e-3)
    rp, rm, rv = adamw_ref(p0, g, m0, v0, 3, 5e-3)
    assert normwise(host(p) - p0, rp - p0) < TOL_FP32
    assert normwise(host(m), rm) < TOL_FP32
    assert normwise(host(v), rv) < TOL_FP32
