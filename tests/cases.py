"""Seeded test problems shared by the GPU parity tests (data only: the
oracle and the HIP path each compute from these arrays)."""
import numpy as np
import torch

from paper_2308_13137_amd import inputs
from paper_2308_13137_amd.configs import Linear, Site, Workload, llama_block


def bf16_exact(a):
    """Round to bf16 storage (the dtype conversion of the inputs)."""
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).float().numpy()


def dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dtype).contiguous()


def small_llama(name, hidden, ffn, T, w_bits, group=None, kv=None, let=False, act_bits=16,
                sigma=0.02):
    return llama_block(name, hidden, ffn, w_bits, group=group, kv_dim=kv, let=let,
                       act_bits=act_bits, T=T, w_sigma=sigma, let_init=let)


def make_problem(w: Workload, seed=0, logit="init", bias=False):
    """Host arrays for one calibration step of workload ``w``:
    X per site, W / B / logits per linear, LET s, delta (SmoothQuant/OS+ init
    from the oracle when the workload asks for it, else None)."""
    from oracle.let import let_init
    from oracle.block import fp_target
    cfg = 1000 + seed
    X = []
    for k, s in enumerate(w.sites):
        rng = inputs.rng_for(cfg, 1, k)
        if w.x_recipe == "small":
            x = inputs.small_activations(rng, w.T, s.width)
        else:
            x = inputs.activations(rng, w.T, s.width)
        X.append(bf16_exact(x) if w.bf16 else x)
    W, B, gl, bl = [], [], [], []
    for l, lin in enumerate(w.linears):
        rng = inputs.rng_for(cfg, 2, l)
        c_in = w.sites[lin.site].width
        wt = inputs.weights(rng, lin.c_out, c_in, w.w_sigma, w.w_outlier)
        W.append(bf16_exact(wt) if w.bf16 else wt)
        B.append(rng.standard_normal(lin.c_out).astype(np.float32) * 0.1 if bias else None)
        ng = c_in // lin.group
        if logit == "init":
            gl.append(np.full((lin.c_out, ng), 4.0, np.float32))
            bl.append(np.full((lin.c_out, ng), 4.0, np.float32))
        else:
            gl.append(rng.uniform(0.5, 5.0, (lin.c_out, ng)).astype(np.float32))
            bl.append(rng.uniform(0.5, 5.0, (lin.c_out, ng)).astype(np.float32))
    s, d = [], []
    for k, site in enumerate(w.sites):
        if site.let:
            Ws = [W[l] for l, lin in enumerate(w.linears) if lin.site == k]
            sk, dk = let_init(X[k], Ws)
            s.append(sk)
            d.append(dk)
        else:
            s.append(None)
            d.append(None)
    Y = [fp_target(X[lin.site], W[l], B[l], bf16=w.bf16) for l, lin in enumerate(w.linears)]
    return dict(X=X, W=W, B=B, gamma_logit=gl, beta_logit=bl, s=s, delta=d, Y=Y)


def normwise(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / den) if den > 0 else float(np.max(np.abs(got)))
