"""The allocation-free activation backward (oq_act_fakequant_bwd_noalloc)
against the workspace entry point it shares its kernels with.

Two calls in a row on one stream, the second on a smaller input, so the
second reuses the static device scratch the first one wrote; each must equal
oq_act_fakequant_bwd bit for bit (same kernels, same fixed reduction order).
A size whose partials exceed the scratch is refused before any launch."""
import numpy as np
import pytest
import torch

from paper_2308_13137_amd import inputs, oq
from tests.cases import bf16_exact, dev

pytestmark = pytest.mark.gpu


def _case(T, Cw, bits, seed):
    rng = inputs.rng_for(77, seed, T, Cw)
    X = dev(bf16_exact(inputs.activations(rng, T, Cw)), torch.bfloat16)
    s = dev(rng.uniform(0.3, 3.0, Cw).astype(np.float32))
    d = dev((rng.standard_normal(Cw) * 0.2).astype(np.float32))
    G = dev(rng.standard_normal((T, Cw)).astype(np.float32))
    return X, s, d, G, bits


def _both(X, s, d, G, bits):
    T, Cw = X.shape
    ref = oq.act_fakequant_bwd(X, bits, G, s=s, delta=d)
    gx = torch.full((T, Cw), float("nan"), device="cuda")
    ds = torch.full((Cw,), float("nan"), device="cuda")
    dd = torch.full((Cw,), float("nan"), device="cuda")
    oq.act_fakequant_bwd_noalloc_into(X, bits, G, gx, ds, dd, s=s, delta=d)
    return ref, (gx, ds, dd)


def test_noalloc_matches_workspace_entry_twice():
    big = _case(3000, 4096, 4, 0)          # 768 partial rows x 4096 columns
    small = _case(200, 1024, 3, 1)         # smaller: reuses the first call's scratch
    for name, case in (("large", big), ("small", small)):
        print(f"noalloc act_bwd {name} T={case[0].shape[0]} C={case[0].shape[1]}", flush=True)
        ref, got = _both(*case)
        torch.cuda.synchronize()
        for r, g, what in zip(ref, got, ("dX_tilde", "d_s", "d_delta")):
            assert torch.equal(r, g), (name, what)


def test_noalloc_rejects_oversized_partials():
    X, s, d, G, bits = _case(1000, 11008, 4, 2)   # 500 partial rows x 11008 > 32 MiB
    out = torch.empty(11008, device="cuda")
    with pytest.raises(oq.OQError, match="UNSUPPORTED"):
        oq.act_fakequant_bwd_noalloc_into(X, bits, G, None, out, None, s=s, delta=d)
    # without the LET gradients nothing goes to the scratch, so any size runs
    gx = torch.empty_like(G)
    oq.act_fakequant_bwd_noalloc_into(X, bits, G, gx, None, None, s=s, delta=d)
    ref, _, _ = oq.act_fakequant_bwd(X, bits, G, s=s, delta=d)
    torch.cuda.synchronize()
    assert torch.equal(gx, ref)
