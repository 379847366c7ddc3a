"""Host-only checks of the C ABI: the library loads, exports every entry point
declared in include/oq.h, and rejects invalid arguments before it launches
anything (no GPU needed: every call here fails validation or only sizes a
workspace)."""
import ctypes as C
import os
import re

import pytest

from paper_2308_13137_amd import configs, oq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oq.h")

pytestmark = pytest.mark.skipif(not os.path.exists(oq.LIB_PATH), reason="liboq.so not built")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = C.c_void_p(0x10000)      # aligned, never dereferenced: validation fails first
MISALIGNED = C.c_void_p(0x10004)


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oq_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    syms = declared_symbols()
    assert len(syms) >= 20
    L = oq.lib()
    for s in syms:
        assert hasattr(L, s), s
    assert set(syms) == set(oq.SIGNATURES), set(syms) ^ set(oq.SIGNATURES)


def test_status_strings():
    L = oq.lib()
    assert L.oq_status_str(0) == b"OQ_OK"
    assert L.oq_status_str(3) == b"OQ_ERR_WORKSPACE"
    assert L.oq_version() >= 1


def lwc_fwd(**kw):
    a = dict(W=FAKE, w_dt=oq.OQ_BF16, c_out=64, c_in=256, s=None, gl=FAKE, bl=FAKE, bits=4,
             group=64, W_dq=FAKE, dq_dt=oq.OQ_BF16, codes=None, h=None, z=None, st=None)
    a.update(kw)
    return oq.lib().oq_lwc_fakequant_fwd(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(W=None), INVALID), (dict(gl=None), INVALID), (dict(bits=9), UNSUPPORTED),
    (dict(bits=1), UNSUPPORTED), (dict(group=48, c_in=384), UNSUPPORTED), (dict(group=100), INVALID),
    (dict(c_in=252, group=4), INVALID), (dict(W=MISALIGNED), INVALID), (dict(w_dt=7), INVALID),
    (dict(group=1024, c_in=2048), UNSUPPORTED), (dict(c_out=-1), INVALID),
])
def test_lwc_fwd_rejects(kw, status):
    assert lwc_fwd(**kw) == status
    assert oq.lib().oq_last_error()


def test_lwc_bwd_workspace_contract():
    L = oq.lib()
    n = C.c_size_t(0)
    assert L.oq_lwc_fakequant_bwd_workspace_size(4096, 4096, 4096, 1, C.byref(n)) == OK
    assert n.value >= 4096 * 4
    assert L.oq_lwc_fakequant_bwd_workspace_size(4096, 4096, 128, 0, C.byref(n)) == OK
    assert n.value == 0
    # d_s wanted but no workspace: refused before launch
    st = L.oq_lwc_fakequant_bwd(FAKE, oq.OQ_BF16, 64, 256, None, FAKE, FAKE, 4, 64, FAKE, FAKE,
                                FAKE, FAKE, None, None, 0, None)
    assert st == WORKSPACE


def test_act_rejects():
    L = oq.lib()
    assert L.oq_act_fakequant_fwd(FAKE, oq.OQ_BF16, 16, 256, 9, None, None, FAKE, oq.OQ_BF16,
                                  None, None, None, None) == UNSUPPORTED
    assert L.oq_act_fakequant_fwd(FAKE, oq.OQ_BF16, 16, 250, 4, None, None, FAKE, oq.OQ_BF16,
                                  None, None, None, None) == INVALID
    assert L.oq_act_fakequant_bwd(FAKE, oq.OQ_BF16, 16, 256, 4, None, None, FAKE, None, FAKE,
                                  FAKE, None, 0, None) == WORKSPACE


def test_packed_rejects():
    L = oq.lib()
    # pack: bits, shape, alignment
    assert L.oq_pack_codes(FAKE, 4, 64, 9, FAKE, None) == UNSUPPORTED
    assert L.oq_pack_codes(FAKE, 4, 48, 4, FAKE, None) == INVALID
    assert L.oq_pack_codes(MISALIGNED, 4, 64, 4, FAKE, None) == INVALID
    assert L.oq_pack_codes(None, 4, 64, 4, FAKE, None) == INVALID

    def lin(**kw):
        a = dict(X=FAKE, x_dt=oq.OQ_BF16, n_tok=1, c_in=256, P=FAKE, bits=4, group=128, h=FAKE,
                 z=FAKE, B=None, c_out=64, Y=FAKE, y_dt=oq.OQ_F32, st=None)
        a.update(kw)
        return L.oq_packed_linear(*a.values())

    assert lin(x_dt=oq.OQ_F32) == UNSUPPORTED
    assert lin(bits=8) == UNSUPPORTED and lin(bits=1) == UNSUPPORTED
    assert lin(c_in=131072, group=128) == UNSUPPORTED
    assert lin(c_in=240, group=48) == INVALID          # c_in % 32
    assert lin(group=96) == INVALID                     # does not divide 256
    assert lin(group=16, c_in=256) == INVALID           # not a multiple of 32
    assert lin(h=None) == INVALID and lin(z=MISALIGNED) == INVALID
    assert lin(n_tok=-1) == INVALID and lin(y_dt=5) == INVALID
    assert oq.lib().oq_last_error()


def _desc(w):
    d = oq.BlockDesc()
    d.tokens = w.T
    d.n_sites, d.n_linears = len(w.sites), len(w.linears)
    d.dtype = oq.OQ_BF16 if w.bf16 else oq.OQ_F32
    for k, s in enumerate(w.sites):
        d.site_width[k], d.site_let[k], d.site_act_bits[k] = s.width, int(s.let), s.act_bits
    for l, lin in enumerate(w.linears):
        d.lin_site[l], d.lin_c_out[l], d.lin_bits[l], d.lin_group[l] = lin.site, lin.c_out, lin.bits, lin.group
    return d


@pytest.mark.parametrize("w", configs.CONFIGS, ids=[c.name for c in configs.CONFIGS])
def test_block_workspace_sizes(w):
    n = C.c_size_t(0)
    assert oq.lib().oq_block_workspace_size(C.byref(_desc(w)), C.byref(n)) == OK
    T = w.T
    es = 2 if w.bf16 else 4
    biggest = max(sum(l.c_out for l in w.linears if l.site == k) for k in range(len(w.sites)))
    # at least the largest stacked dY^T of one site, and not much more than
    # that: the token-sized buffers are that dY^T, X^ and the LET input
    # gradient, the rest scales with the weights
    assert n.value >= biggest * T * es
    assert n.value < 2 * biggest * T * es + 8 * 2 ** 30


def test_block_desc_validation():
    L = oq.lib()
    n = C.c_size_t(0)
    d = _desc(configs.C2)
    d.lin_site[3] = 3                     # o_proj moved after down_proj's site: not consecutive
    d.lin_site[6] = 1
    assert L.oq_block_workspace_size(C.byref(d), C.byref(n)) == INVALID
    d = _desc(configs.C2)
    d.tokens = 100
    assert L.oq_block_workspace_size(C.byref(d), C.byref(n)) == INVALID
    d = _desc(configs.C2)
    d.lin_bits[0] = 1
    assert L.oq_block_workspace_size(C.byref(d), C.byref(n)) == UNSUPPORTED
    d = _desc(configs.C2)
    d.site_act_bits[0] = 12
    assert L.oq_block_workspace_size(C.byref(d), C.byref(n)) == UNSUPPORTED
    # a step with too small a workspace is refused before any launch
    prm, grd = oq.BlockParams(), oq.BlockGrads()
    d = _desc(configs.C1)
    prm.W[0] = prm.gamma_logit[0] = prm.beta_logit[0] = 0x10000
    grd.d_gamma_logit[0] = grd.d_beta_logit[0] = 0x10000
    yp = (C.c_void_p * 1)(0x10000)
    xp = (C.c_void_p * 1)(0x10000)
    st = L.oq_block_calib_step(C.byref(d), yp, xp, C.byref(prm), C.byref(grd), None, FAKE, FAKE,
                               16, None)
    assert st == WORKSPACE


def _export_call(d, prm=None, packed=None, h=None, z=None, ws=FAKE, nbytes=None):
    L = oq.lib()
    n = C.c_size_t(0)
    L.oq_block_export_workspace_size(C.byref(d), C.byref(n))
    nl = d.n_linears
    arr = lambda v: (C.c_void_p * nl)(*([v] * nl))
    if prm is None:
        prm = oq.BlockParams()
        for l in range(nl):
            prm.W[l] = prm.gamma_logit[l] = prm.beta_logit[l] = 0x10000
        for k in range(d.n_sites):
            prm.s[k] = prm.delta[k] = 0x10000
    return L.oq_block_export(C.byref(d), C.byref(prm), packed or arr(0x10000), h or arr(0x10000),
                             z or arr(0x10000), None, ws, n.value if nbytes is None else nbytes,
                             None)


def test_export_validation():
    """oq_block_export checks everything before its first launch: workspace
    size and alignment, C_in % 32, outputs, and that the packed linear can
    consume what it writes (bits 2..7, groups of whole 32-code runs)."""
    L = oq.lib()
    assert _export_call(_desc(configs.C2), nbytes=16) == WORKSPACE
    assert _export_call(_desc(configs.C2), ws=MISALIGNED) == WORKSPACE
    assert _export_call(_desc(configs.C2), ws=None) == WORKSPACE
    d = _desc(configs.C2)
    d.lin_bits[2] = 8
    assert _export_call(d) == UNSUPPORTED and b"packed_linear" in L.oq_last_error()
    d = _desc(configs.C2)
    for l in range(d.n_linears):
        d.lin_group[l] = 16
    assert _export_call(d) == UNSUPPORTED
    d = _desc(configs.C1)
    d.site_width[0] = d.lin_c_out[0] = 264          # C_in % 32 != 0 (groups of 8 divide it)
    d.lin_group[0] = 8
    assert _export_call(d) == INVALID
    nl = configs.C2.linears
    missing = (C.c_void_p * len(nl))(*([0x10000] * (len(nl) - 1) + [None]))
    assert _export_call(_desc(configs.C2), packed=missing) == INVALID
    assert _export_call(_desc(configs.C2), z=missing) == INVALID
    misaligned = (C.c_void_p * len(nl))(*([0x10004] * len(nl)))
    assert _export_call(_desc(configs.C2), packed=misaligned) == INVALID


def test_block_plan_of_benchmark_workloads():
    """The launch plan is a host-side function of the descriptor: at the
    benchmark's 262,144 tokens every site runs in sequence and the gradient
    products read their operands as stored; the plans the full-size GPU tests
    assert are the ones fixed here."""
    L = oq.lib()
    expect = {  # per site: concurrent, direct, wgrad splits, fwd splits, fused LWC bwd, W^T copy
        "llama7b_w3a16_g128": [[0, 1, 1, 1, 1, 0], [0, 1, 1, 1, 1, 0], [0, 1, 2, 1, 0, 0], [0, 1, 4, 1, 0, 0]],
        "llama7b_w4a4_let_lwc": [[0, 1, 1, 1, 0, 1], [0, 1, 1, 1, 0, 1], [0, 1, 2, 1, 0, 1], [0, 1, 4, 1, 0, 0]],
        "llama13b_w2a16_g64": [[0, 1, 4, 1, 0, 0], [0, 1, 8, 1, 0, 0], [0, 1, 2, 1, 0, 0], [0, 1, 4, 1, 0, 0]],
        "llama2_70b_w4a16_g128": [[0, 1, 1, 1, 1, 0]] * 4,
    }
    for w in configs.CONFIGS[1:]:
        n = 6 * len(w.sites)
        buf = (C.c_int * n)()
        assert L.oq_block_plan(C.byref(_desc(w)), buf, n) == OK
        assert [list(buf[i * 6:(i + 1) * 6]) for i in range(len(w.sites))] == expect[w.name], w.name
    # the paper's 2048-token segment runs the sites concurrently
    buf = (C.c_int * 24)()
    assert L.oq_block_plan(C.byref(_desc(configs.C2.with_tokens(2048))), buf, 24) == OK
    assert all(buf[6 * k] == 1 for k in range(4))
    assert L.oq_block_plan(C.byref(_desc(configs.C2)), buf, 5) == INVALID


def test_calibrate_validation():
    L = oq.lib()
    d = _desc(configs.C1)
    n = C.c_size_t(0)
    assert L.oq_block_workspace_size(C.byref(d), C.byref(n)) == OK
    prm, grd, opt = oq.BlockParams(), oq.BlockGrads(), oq.BlockOptim()
    opt.step = 1
    yp = (C.c_void_p * 2)(0x10000, None)           # segment 1's target missing
    xp = (C.c_void_p * 2)(0x10000, 0x10000)
    args = lambda **kw: dict(dict(nseg=2, ep=2, yp=yp, xp=xp, losses=FAKE, ws=FAKE, nbytes=n.value),
                             **kw)

    def call(**kw):
        a = args(**kw)
        return L.oq_block_calibrate(C.byref(d), a["nseg"], a["ep"], a["yp"], a["xp"], C.byref(prm),
                                    C.byref(grd), C.byref(opt), a["losses"], a["ws"], a["nbytes"],
                                    None)

    assert call() == INVALID                        # found before any launch
    assert call(nseg=0) == INVALID and call(ep=0) == INVALID
    assert call(losses=None) == INVALID
    assert call(nbytes=n.value - 1) == WORKSPACE
    opt.step = 0
    assert call() == INVALID


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(oq, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(oq, "_lib", None)
    with pytest.raises(oq.OQError):
        oq.lib()


def test_act_bwd_noalloc_limits():
    """The allocation-free activation backward refuses, before any launch,
    sizes whose column partials exceed its static scratch, and bad pointers."""
    L = oq.lib()
    lim = 32 * 1024 * 1024
    n = C.c_size_t(0)
    assert L.oq_act_fakequant_bwd_workspace_size(1000, 11008, C.byref(n)) == OK
    assert n.value > lim
    assert L.oq_act_fakequant_bwd_noalloc(FAKE, oq.OQ_BF16, 1000, 11008, 4, None, None, FAKE,
                                          None, FAKE, None, None) == UNSUPPORTED
    assert b"scratch" in L.oq_last_error()
    assert L.oq_act_fakequant_bwd_noalloc(FAKE, oq.OQ_BF16, 1000, 11008, 4, None, None, MISALIGNED,
                                          None, FAKE, None, None) == INVALID
    assert L.oq_act_fakequant_bwd_noalloc(FAKE, oq.OQ_BF16, 16, 256, 9, None, None, FAKE,
                                          None, FAKE, None, None) == UNSUPPORTED
    assert L.oq_act_fakequant_bwd_workspace_size(1 << 20, 4096, C.byref(n)) == OK
    assert n.value <= lim        # 4096 channels fit at any token count


def _ckpt_bytes(w, completed=3, c_out_override=None, bad_hash=False, truncate=0):
    """A checkpoint file written by hand from the layout include/oq.h states
    (no AdamW state): header, shape record, then each clipping-logit tensor."""
    import struct
    import numpy as np
    nl, ns = len(w.linears), len(w.sites)
    pad = lambda xs, n: list(xs) + [0] * (n - len(xs))
    c_outs = [l.c_out for l in w.linears]
    if c_out_override is not None:
        c_outs[0] = c_out_override
    shape = struct.pack("<ii8q8i8i16i16q16i16q16i", ns, nl,
                        *pad([s.width for s in w.sites], 8), *pad([int(s.let) for s in w.sites], 8),
                        *pad([s.act_bits for s in w.sites], 8), *pad([l.site for l in w.linears], 16),
                        *pad(c_outs, 16), *pad([l.bits for l in w.linears], 16),
                        *pad([l.group for l in w.linears], 16), *pad([0] * nl, 16))
    assert len(shape) == 584
    tensors = []
    for i, l in enumerate(w.linears):
        n = l.c_out * (w.sites[l.site].width // l.group)
        for kind in (0, 1):
            data = np.full(n, 4.0, np.float32).tobytes()
            h = 1469598103934665603
            for byte in data:
                h = ((h ^ byte) * 1099511628211) & (2 ** 64 - 1)
            if bad_hash:
                h ^= 1
            tensors.append(struct.pack("<IIQQ", kind, i, n, h) + data)
    head = b"OQCKPT\0\1" + struct.pack("<iiii", 1, 584, completed, 0) + shape + \
        struct.pack("<Q", len(tensors))
    blob = head + b"".join(tensors)
    return blob[:len(blob) - truncate] if truncate else blob


def test_checkpoint_load_validation(tmp_path):
    """A block checkpoint is verified completely before any device buffer is
    written: magic, shape, sizes and every hash (the file is written here
    from the documented layout)."""
    L = oq.lib()
    w = configs.C1
    d = _desc(w)
    prm = oq.BlockParams()
    prm.W[0] = prm.gamma_logit[0] = prm.beta_logit[0] = 0x10000
    done = C.c_int(-1)

    def load(blob):
        p = tmp_path / "ck.bin"
        p.write_bytes(blob)
        return L.oq_block_state_load(C.byref(d), C.byref(prm), None, C.byref(done),
                                     str(p).encode(), None)
    assert load(b"NOTACKPT" + _ckpt_bytes(w)[8:]) == INVALID
    assert b"not a block checkpoint" in L.oq_last_error()
    assert load(_ckpt_bytes(w, c_out_override=128)) == INVALID
    assert b"shape" in L.oq_last_error()
    assert load(_ckpt_bytes(w, bad_hash=True)) == INVALID
    assert b"checksum" in L.oq_last_error()
    assert load(_ckpt_bytes(w, truncate=100)) == INVALID
    assert b"truncated" in L.oq_last_error()
    assert L.oq_block_state_load(C.byref(d), C.byref(prm), None, C.byref(done),
                                 str(tmp_path / "missing.bin").encode(), None) == INVALID
    assert done.value == -1                      # nothing reported on failure


def _llama_desc(softmax_bits=16):
    d = oq.LlamaDesc()
    d.tokens, d.seq_len, d.hidden, d.ffn, d.heads, d.kv_heads = 128, 128, 256, 512, 2, 1
    d.norm_eps, d.rope_base = 1e-6, 10000.0
    for l in range(7):
        d.w_bits[l], d.w_group[l] = 4, 128
    d.act_bits, d.let, d.softmax_bits = 16, 0, softmax_bits
    return d


def test_llama_softmax_bits_and_attention_validation():
    L = oq.lib()
    n = C.c_size_t(0)
    assert L.oq_llama_workspace_size(C.byref(_llama_desc(4)), C.byref(n)) == OK
    n16 = C.c_size_t(0)
    assert L.oq_llama_workspace_size(C.byref(_llama_desc(16)), C.byref(n16)) == OK
    assert n.value > n16.value                      # the per-row record and the larger scratch
    for bad in (1, 9, 15):
        assert L.oq_llama_workspace_size(C.byref(_llama_desc(bad)), C.byref(n)) == UNSUPPORTED
    ws = C.c_size_t(0)
    assert L.oq_attention_bwd_workspace_size(128, 2, 4, C.byref(ws)) == OK
    assert ws.value == 3 * 128 * 2 * 4 + 256
    assert L.oq_attention_bwd_workspace_size(128, 2, 16, C.byref(ws)) == OK
    assert ws.value == 128 * 2 * 4 + 256

    def fwd(bits, pstat):
        return L.oq_attention_fwd(FAKE, FAKE, FAKE, 128, 64, 2, 1, 64, bits, FAKE, FAKE, pstat, None)
    assert fwd(4, None) == INVALID and fwd(4, MISALIGNED) == INVALID
    assert fwd(9, FAKE) == INVALID and fwd(1, FAKE) == INVALID

    def bwd(bits, pstat, nbytes):
        return L.oq_attention_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, pstat, 128, 64, 2, 1, 64, bits, FAKE,
                                  FAKE, FAKE, FAKE, nbytes, None)
    assert bwd(4, None, 1 << 20) == INVALID
    assert bwd(4, FAKE, 3 * 128 * 2 * 4) == WORKSPACE     # one fp32 [H, T] short of the three


def test_llama_calibrate_validation():
    L = oq.lib()
    d = _llama_desc()
    n = C.c_size_t(0)
    assert L.oq_llama_workspace_size(C.byref(d), C.byref(n)) == OK
    prm, grd, opt = oq.LlamaParams(), oq.LlamaGrads(), oq.LlamaOptim()
    opt.step = 1
    hp = (C.c_void_p * 2)(0x10000, 0x10000)
    tp = (C.c_void_p * 2)(0x10000, None)           # sample 1's target missing

    def call(ns=2, ep=2, h=hp, t=tp, losses=FAKE):
        return L.oq_llama_calibrate(C.byref(d), ns, ep, h, t, C.byref(prm), C.byref(grd),
                                    C.byref(opt), losses, FAKE, n.value, None)
    assert call() == INVALID                        # found before any launch
    assert call(ns=0) == INVALID and call(ep=0) == INVALID
    assert call(losses=None) == INVALID
    assert call(t=(C.c_void_p * 2)(0x10000, 0x10004)) == INVALID     # misaligned
    opt.step = 0
    assert call(t=(C.c_void_p * 2)(0x10000, 0x10000)) == INVALID
