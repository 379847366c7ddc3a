"""Seeded synthetic inputs for the calibration step.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic.  The same recipes exist for numpy (host, small cases)
and for torch on a device (full-size workloads, where drawing on the host
would take minutes).  The two backends draw from different streams; a test
that needs identical bytes on both sides draws once and copies.

Recipes (stand-ins for WikiText2 activations and LLaMA weights, which are
not available here):
  weights      N(0, sigma); a fraction ``outlier_frac`` of entries, chosen
               uniformly without replacement, multiplied by ``outlier_mult``
  activations  per site, round(outlier_frac * C) channels drawn as
               outlier_mult * Student-t(dof), the rest N(0, 1); each token
               row then divided by its root-mean-square (unit-gain RMSNorm)
  small case   X ~ N(0, 1) with ``n_outlier`` channels multiplied by 20
"""
import numpy as np

SEED = 20230825


def rng_for(*key):
    """A numpy Generator keyed by (config, tensor, index...) integers."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, *key])))


def weights(rng, c_out, c_in, sigma, outlier_frac=0.0, outlier_mult=10.0):
    w = rng.standard_normal((c_out, c_in), dtype=np.float32) * np.float32(sigma)
    n_out = int(round(outlier_frac * c_out * c_in))
    if n_out:
        idx = rng.choice(c_out * c_in, size=n_out, replace=False)
        w.reshape(-1)[idx] *= np.float32(outlier_mult)
    return w


def activations(rng, T, C, outlier_frac=0.01, outlier_mult=10.0, dof=3, rms_norm=True):
    x = rng.standard_normal((T, C), dtype=np.float32)
    n_ch = int(round(outlier_frac * C))
    if n_ch:
        ch = rng.choice(C, size=n_ch, replace=False)
        z = rng.standard_normal((T, n_ch))
        chi2 = np.sum(rng.standard_normal((dof, T, n_ch)) ** 2, axis=0)
        x[:, ch] = (outlier_mult * z / np.sqrt(chi2 / dof)).astype(np.float32)
    if rms_norm:
        x /= np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=1, keepdims=True) + 1e-6).astype(np.float32)
    return x


def small_activations(rng, T, C, n_outlier=4, mult=20.0):
    x = rng.standard_normal((T, C), dtype=np.float32)
    ch = rng.choice(C, size=n_outlier, replace=False)
    x[:, ch] *= np.float32(mult)
    return x


# ---------------------------------------------------------------- torch (device)
def torch_weights(gen, c_out, c_in, sigma, outlier_frac=0.0, outlier_mult=10.0,
                  device="cuda", dtype=None):
    import torch
    w = torch.randn((c_out, c_in), generator=gen, device=device, dtype=torch.float32) * sigma
    n_out = int(round(outlier_frac * c_out * c_in))
    if n_out:
        idx = torch.randperm(c_out * c_in, generator=gen, device=device)[:n_out]
        w.view(-1)[idx] *= outlier_mult
    return w if dtype is None else w.to(dtype)


def torch_activations(gen, T, C, outlier_frac=0.01, outlier_mult=10.0, dof=3,
                      device="cuda", dtype=None, chunk=16384):
    """Drawn in token chunks so the fp32 temporary stays small."""
    import torch
    out = torch.empty((T, C), device=device, dtype=dtype or torch.float32)
    n_ch = int(round(outlier_frac * C))
    ch = torch.randperm(C, generator=gen, device=device)[:n_ch]
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        x = torch.randn((t1 - t0, C), generator=gen, device=device, dtype=torch.float32)
        if n_ch:
            z = torch.randn((t1 - t0, n_ch), generator=gen, device=device)
            chi2 = (torch.randn((dof, t1 - t0, n_ch), generator=gen, device=device) ** 2).sum(0)
            x[:, ch] = outlier_mult * z / torch.sqrt(chi2 / dof)
        x /= torch.sqrt(x.double().pow(2).mean(1, keepdim=True) + 1e-6).float()
        out[t0:t1] = x
    return out
