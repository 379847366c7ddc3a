"""The calibration workloads: shapes, bit widths, group sizes and input recipes.

A block is described by its input sites and its linears.  A site is one
input tensor shared by the linears that read it (for a LLaMA block: the
q/k/v input, the o_proj input, the gate/up input and the down_proj input).
LET, when on, scales and shifts the first three sites; the FFN's second
linear has none (Sec. 3.3 "Linear layer": every linear except the FFN's
second).
"""
from dataclasses import dataclass, field, replace
from typing import List, Optional


@dataclass(frozen=True)
class Site:
    width: int
    let: bool = False
    act_bits: int = 16          # 16 = activations stay in full precision


@dataclass(frozen=True)
class Linear:
    name: str
    site: int
    c_out: int
    bits: int
    group: int                  # contiguous input channels per quantisation group


@dataclass(frozen=True)
class Workload:
    name: str
    T: int                      # tokens per calibration step
    sites: List[Site]
    linears: List[Linear]
    bf16: bool = True           # bf16 storage + bf16 matrix cores; else fp32 throughout
    w_sigma: float = 0.02
    w_outlier: float = 0.001
    x_recipe: str = "llm"       # "llm" (outlier channels + RMSNorm) or "small"
    steps: int = 1
    let_init: bool = False      # SmoothQuant / OS+ initialisation of s, delta
    description: str = ""

    def with_tokens(self, T):
        return replace(self, T=T)

    def oracle_desc(self):
        """The plain-dict description the oracle takes."""
        return dict(T=self.T, bf16=self.bf16,
                    sites=[dict(width=s.width, let=s.let, act_bits=s.act_bits) for s in self.sites],
                    linears=[dict(site=l.site, c_out=l.c_out, bits=l.bits, group=l.group)
                             for l in self.linears])

    def c_in(self, l):
        return self.sites[self.linears[l].site].width

    @property
    def n_params(self):
        return sum(l.c_out * self.sites[l.site].width for l in self.linears)


def llama_block(name, hidden, ffn, w_bits, group=None, kv_dim=None, let=False,
                act_bits=16, T=128 * 2048, **kw):
    """The seven linears of a LLaMA block.  ``group=None`` = per output channel."""
    kv = kv_dim or hidden
    g_h = group or hidden
    g_f = group or ffn
    sites = [Site(hidden, let, act_bits), Site(hidden, let, act_bits),
             Site(hidden, let, act_bits), Site(ffn, False, act_bits)]
    lins = [Linear("q_proj", 0, hidden, w_bits, g_h), Linear("k_proj", 0, kv, w_bits, g_h),
            Linear("v_proj", 0, kv, w_bits, g_h), Linear("o_proj", 1, hidden, w_bits, g_h),
            Linear("gate_proj", 2, ffn, w_bits, g_h), Linear("up_proj", 2, ffn, w_bits, g_h),
            Linear("down_proj", 3, hidden, w_bits, g_f)]
    return Workload(name=name, T=T, sites=sites, linears=lins, **kw)


C1 = Workload(
    name="linear256_w4a16_g64_fp32", T=128,
    sites=[Site(256)], linears=[Linear("linear", 0, 256, 4, 64)],
    bf16=False, w_sigma=0.02, w_outlier=0.0, x_recipe="small",
    description="one 256x256 linear, W4A16 LWC g64, fp32, 128 tokens")

C2 = llama_block("llama7b_w3a16_g128", 4096, 11008, w_bits=3, group=128,
                 description="LLaMA-7B-shaped block linears, W3A16 LWC g128, bf16, 128x2048 tokens")

C3 = llama_block("llama7b_w4a4_let_lwc", 4096, 11008, w_bits=4, group=None, let=True,
                 act_bits=4, let_init=True,
                 description="LLaMA-7B-shaped block linears, W4A4 LET+LWC, per-channel weights, "
                             "per-token activations, bf16, 128x2048 tokens")

C4 = llama_block("llama13b_w2a16_g64", 5120, 13824, w_bits=2, group=64, steps=20,
                 description="LLaMA-13B-shaped block linears, W2A16 LWC g64, bf16, 20 steps")

C5 = llama_block("llama2_70b_w4a16_g128", 8192, 28672, w_bits=4, group=128, kv_dim=1024,
                 w_sigma=0.015,
                 description="LLaMA-2-70B-shaped block linears (GQA k/v 1024), W4A16 LWC g128, bf16")

CONFIGS = [C1, C2, C3, C4, C5]
BY_NAME = {c.name: c for c in CONFIGS}
