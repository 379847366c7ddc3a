"""Thin Python binding of liboq.so (declared in include/oq.h).

Every function here only marshals arguments: it checks dtypes and devices,
allocates output tensors with torch (device memory is torch's job) and calls
the C entry point of the same name on the current HIP stream.  All arithmetic
happens in the library's HIP kernels.  If ``liboq.so`` has not been built the
first call raises :class:`OQError`; there is no fallback.
"""
import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboq.so")

OQ_F32, OQ_BF16 = 0, 1
WQ_LWC, WQ_PACT, WQ_LSQ = 0, 1, 2          # weight quantisers (lin_quant)
ACT_SYM = 0x100                            # OR into activation bits: symmetric absmax
MAX_SITES, MAX_LINEARS = 8, 16
PROF_KINDS = ["gemm_fwd", "gemm_wgrad", "gemm_dgrad", "lwc_fwd", "lwc_bwd", "act_fwd",
              "act_bwd", "transpose", "other", "packed_linear", "attn_fwd", "attn_bwd"]

# name -> (restype, argtypes); the exported surface of include/oq.h
_P, _I64, _I, _D, _SZ = C.c_void_p, C.c_int64, C.c_int, C.c_double, C.c_size_t
_PSZ = C.POINTER(C.c_size_t)
SIGNATURES = {
    "oq_status_str": (C.c_char_p, [_I]),
    "oq_last_error": (C.c_char_p, []),
    "oq_version": (_I, []),
    "oq_lwc_fakequant_fwd": (_I, [_P, _I, _I64, _I64, _P, _P, _P, _I, _I64, _P, _I, _P, _P, _P, _P]),
    "oq_lwc_fakequant_bwd": (_I, [_P, _I, _I64, _I64, _P, _P, _P, _I, _I64, _P, _P, _P, _P, _P,
                                  _P, _SZ, _P]),
    "oq_lwc_fakequant_bwd_workspace_size": (_I, [_I64, _I64, _I64, _I, _PSZ]),
    "oq_wquant_fakequant_fwd": (_I, [_I, _P, _I, _I64, _I64, _P, _P, _P, _I, _I64, _P, _I, _P, _P,
                                     _P, _P]),
    "oq_wquant_fakequant_bwd": (_I, [_I, _P, _I, _I64, _I64, _P, _P, _P, _I, _I64, _P, _P, _P, _P,
                                     _P, _P, _SZ, _P]),
    "oq_wquant_init": (_I, [_I, _P, _I, _I64, _I64, _P, _I, _I64, _P, _P, _P]),
    "oq_let_fold": (_I, [_P, _I, _P, _I64, _I64, _P, _P, _P, _I, _P, _P]),
    "oq_act_fakequant_fwd": (_I, [_P, _I, _I64, _I64, _I, _P, _P, _P, _I, _P, _P, _P, _P]),
    "oq_act_fakequant_bwd": (_I, [_P, _I, _I64, _I64, _I, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_act_fakequant_bwd_workspace_size": (_I, [_I64, _I64, _PSZ]),
    "oq_act_fakequant_bwd_noalloc": (_I, [_P, _I, _I64, _I64, _I, _P, _P, _P, _P, _P, _P, _P]),
    "oq_let_init": (_I, [_P, _I, _I64, _I64, _P, _P, _I, _I, _P, _P, _P, _SZ, _P]),
    "oq_let_init_workspace_size": (_I, [_I64, _I64, _P, _I, _PSZ]),
    "oq_fp_target": (_I, [_P, _P, _I, _P, _I64, _I64, _I64, _P, _P]),
    "oq_matmul_nt": (_I, [_P, _P, _I, _I64, _I64, _I64, _P, _I, _P]),
    "oq_matmul": (_I, [_P, _I, _P, _I, _I64, _I64, _I64, _P, _P]),
    "oq_adamw_step": (_I, [_P, _P, _P, _P, _I64, _D, _D, _D, _D, _D, _I, _P]),
    "oq_block_workspace_size": (_I, [_P, _PSZ]),
    "oq_block_plan": (_I, [_P, _P, _I]),
    "oq_block_calib_step": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_block_calibrate": (_I, [_P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_block_export_workspace_size": (_I, [_P, _PSZ]),
    "oq_block_export": (_I, [_P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_let_absorb": (_I, [_P, _I, _P, _I64, _I64, _P, _P, _P, _P, _P]),
    "oq_block_state_save": (_I, [_P, _P, _P, _I, C.c_char_p, _P]),
    "oq_block_state_load": (_I, [_P, _P, _P, C.POINTER(C.c_int), C.c_char_p, _P]),
    "oq_pack_codes": (_I, [_P, _I64, _I64, _I, _P, _P]),
    "oq_packed_linear": (_I, [_P, _I, _I64, _I64, _P, _I, _I64, _P, _P, _P, _I64, _P, _I, _P]),
    "oq_profile_enable": (_I, [_I]),
    "oq_profile_reset": (_I, []),
    "oq_profile_read": (_I, [_I, C.POINTER(C.c_int64), C.POINTER(C.c_double),
                             C.POINTER(C.c_double)]),
}


class OQError(RuntimeError):
    pass


class BlockDesc(C.Structure):
    _fields_ = [("tokens", C.c_int64), ("n_sites", C.c_int), ("n_linears", C.c_int),
                ("dtype", C.c_int),
                ("site_width", C.c_int64 * MAX_SITES), ("site_let", C.c_int * MAX_SITES),
                ("site_act_bits", C.c_int * MAX_SITES), ("lin_site", C.c_int * MAX_LINEARS),
                ("lin_c_out", C.c_int64 * MAX_LINEARS), ("lin_bits", C.c_int * MAX_LINEARS),
                ("lin_group", C.c_int64 * MAX_LINEARS), ("lin_quant", C.c_int * MAX_LINEARS)]


class BlockParams(C.Structure):
    _fields_ = [("W", C.c_void_p * MAX_LINEARS), ("B", C.c_void_p * MAX_LINEARS),
                ("gamma_logit", C.c_void_p * MAX_LINEARS), ("beta_logit", C.c_void_p * MAX_LINEARS),
                ("s", C.c_void_p * MAX_SITES), ("delta", C.c_void_p * MAX_SITES)]


class BlockGrads(C.Structure):
    _fields_ = [("d_gamma_logit", C.c_void_p * MAX_LINEARS),
                ("d_beta_logit", C.c_void_p * MAX_LINEARS),
                ("d_s", C.c_void_p * MAX_SITES), ("d_delta", C.c_void_p * MAX_SITES),
                ("row_loss", C.c_void_p * MAX_LINEARS)]


class BlockOptim(C.Structure):
    _fields_ = [("m_gamma", C.c_void_p * MAX_LINEARS), ("v_gamma", C.c_void_p * MAX_LINEARS),
                ("m_beta", C.c_void_p * MAX_LINEARS), ("v_beta", C.c_void_p * MAX_LINEARS),
                ("m_s", C.c_void_p * MAX_SITES), ("v_s", C.c_void_p * MAX_SITES),
                ("m_delta", C.c_void_p * MAX_SITES), ("v_delta", C.c_void_p * MAX_SITES),
                ("step", C.c_int), ("lr_lwc", C.c_double), ("lr_let", C.c_double),
                ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
                ("wd", C.c_double), ("frozen", C.c_int)]


FREEZE_LWC, FREEZE_LET = 1, 2


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OQError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2308_13137_amd.build`")
        handle = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status):
    if status != 0:
        L = lib()
        raise OQError(f"{L.oq_status_str(status).decode()}: {L.oq_last_error().decode()}")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise OQError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise OQError("tensors must be contiguous")
    return C.c_void_p(t.data_ptr())


def _dt(t):
    if t.dtype == torch.bfloat16:
        return OQ_BF16
    if t.dtype == torch.float32:
        return OQ_F32
    raise OQError(f"unsupported dtype {t.dtype}")


def _tdt(code):
    return torch.bfloat16 if code == OQ_BF16 else torch.float32


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _f32(t, name):
    if t is not None and t.dtype != torch.float32:
        raise OQError(f"{name} must be float32")
    return t


def lwc_fakequant_fwd(W, gamma_logit, beta_logit, bits, group, s=None, dq_dtype=None,
                      codes=True, hz=True, stream=None):
    """Eq. 2 forward.  Returns (W_dq, codes | None, h | None, z | None)."""
    c_out, c_in = W.shape
    ng = c_in // group
    dq_dtype = dq_dtype or W.dtype
    W_dq = torch.empty((c_out, c_in), dtype=dq_dtype, device=W.device)
    cd = torch.empty((c_out, c_in), dtype=torch.uint8, device=W.device) if codes else None
    h = torch.empty((c_out, ng), dtype=torch.float32, device=W.device) if hz else None
    z = torch.empty((c_out, ng), dtype=torch.float32, device=W.device) if hz else None
    _check(lib().oq_lwc_fakequant_fwd(_ptr(W), _dt(W), c_out, c_in, _ptr(_f32(s, "s")),
                                      _ptr(_f32(gamma_logit, "gamma_logit")),
                                      _ptr(_f32(beta_logit, "beta_logit")), bits, group,
                                      _ptr(W_dq), _dt(W_dq), _ptr(cd), _ptr(h), _ptr(z),
                                      _stream(stream)))
    return W_dq, cd, h, z


def lwc_fakequant_bwd(W, gamma_logit, beta_logit, bits, group, dW_dq, s=None, want_d_s=False,
                      want_dW_tilde=False, stream=None):
    """Straight-through backward.  Returns (d_gamma_logit, d_beta_logit, d_s | None, dW_tilde | None)."""
    c_out, c_in = W.shape
    ng = c_in // group
    dev = W.device
    dg = torch.empty((c_out, ng), dtype=torch.float32, device=dev)
    db = torch.empty((c_out, ng), dtype=torch.float32, device=dev)
    ds = torch.empty(c_in, dtype=torch.float32, device=dev) if want_d_s else None
    dwt = torch.empty((c_out, c_in), dtype=torch.float32, device=dev) if want_dW_tilde else None
    n = C.c_size_t(0)
    _check(lib().oq_lwc_fakequant_bwd_workspace_size(c_out, c_in, group, int(want_d_s), C.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=dev)
    _check(lib().oq_lwc_fakequant_bwd(_ptr(W), _dt(W), c_out, c_in, _ptr(_f32(s, "s")),
                                      _ptr(gamma_logit), _ptr(beta_logit), bits, group,
                                      _ptr(_f32(dW_dq, "dW_dq")), _ptr(dg), _ptr(db), _ptr(ds),
                                      _ptr(dwt), _ptr(ws), n.value, _stream(stream)))
    return dg, db, ds, dwt


def wquant_fakequant_fwd(quantizer, W, p1, p2, bits, group, s=None, dq_dtype=None, codes=True,
                         hz=True, stream=None):
    """Any weight quantiser's forward (WQ_LWC / WQ_PACT / WQ_LSQ).
    Returns (W_dq, codes | None, h | None, z | None)."""
    c_out, c_in = W.shape
    dev = W.device
    dq_dt = _dt(W) if dq_dtype is None else (OQ_BF16 if dq_dtype == torch.bfloat16 else OQ_F32)
    W_dq = torch.empty((c_out, c_in), dtype=_tdt(dq_dt), device=dev)
    cd = torch.empty((c_out, c_in), dtype=torch.uint8, device=dev) if codes else None
    ng = c_in // group
    h = torch.empty((c_out, ng), dtype=torch.float32, device=dev) if hz else None
    z = torch.empty((c_out, ng), dtype=torch.float32, device=dev) if hz else None
    _check(lib().oq_wquant_fakequant_fwd(quantizer, _ptr(W), _dt(W), c_out, c_in, _ptr(s),
                                         _ptr(_f32(p1, "p1")), _ptr(_f32(p2, "p2")), bits, group,
                                         _ptr(W_dq), dq_dt, _ptr(cd), _ptr(h), _ptr(z),
                                         _stream(stream)))
    return W_dq, cd, h, z


def wquant_fakequant_bwd(quantizer, W, p1, p2, bits, group, dW_dq, s=None, want_d_s=False,
                         want_dW_tilde=False, stream=None):
    """Returns (d_p1, d_p2, d_s | None, dW_tilde | None)."""
    c_out, c_in = W.shape
    dev = W.device
    f32 = dict(dtype=torch.float32, device=dev)
    d1 = torch.empty_like(p1)
    d2 = torch.empty_like(p2)
    ds = torch.empty(c_in, **f32) if want_d_s else None
    dwt = torch.empty((c_out, c_in), **f32) if want_dW_tilde else None
    n = C.c_size_t(0)
    _check(lib().oq_lwc_fakequant_bwd_workspace_size(c_out, c_in, group, int(want_d_s), C.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=dev)
    _check(lib().oq_wquant_fakequant_bwd(quantizer, _ptr(W), _dt(W), c_out, c_in, _ptr(s),
                                         _ptr(p1), _ptr(p2), bits, group,
                                         _ptr(_f32(dW_dq, "dW_dq")), _ptr(d1), _ptr(d2), _ptr(ds),
                                         _ptr(dwt), _ptr(ws), n.value, _stream(stream)))
    return d1, d2, ds, dwt


def wquant_init(quantizer, W, bits, group, s=None, stream=None):
    """MinMax starting parameters (p1, p2) of a weight quantiser per group."""
    c_out, c_in = W.shape
    p1 = torch.empty((c_out, c_in // group), dtype=torch.float32, device=W.device)
    p2 = torch.empty_like(p1)
    _check(lib().oq_wquant_init(quantizer, _ptr(W), _dt(W), c_out, c_in, _ptr(s), bits, group,
                                _ptr(p1), _ptr(p2), _stream(stream)))
    return p1, p2


def let_fold(W, B=None, s=None, delta=None, wt_dtype=None, want_W_tilde=True, stream=None):
    """Eq. 3 fold.  Returns (W_tilde | None, B_tilde)."""
    c_out, c_in = W.shape
    wt_dtype = wt_dtype or W.dtype
    Wt = torch.empty((c_out, c_in), dtype=wt_dtype, device=W.device) if want_W_tilde else None
    Bt = torch.empty(c_out, dtype=torch.float32, device=W.device)
    _check(lib().oq_let_fold(_ptr(W), _dt(W), _ptr(_f32(B, "B")), c_out, c_in, _ptr(s), _ptr(delta),
                             _ptr(Wt), OQ_BF16 if wt_dtype == torch.bfloat16 else OQ_F32,
                             _ptr(Bt), _stream(stream)))
    return Wt, Bt


def act_fakequant_fwd(X, bits, s=None, delta=None, dq_dtype=None, codes=True, hz=True,
                      stream=None):
    """Per-token fake-quant of X~ = (X - delta)/s.  Returns (X_dq, codes | None, h | None, z | None)."""
    T, Cw = X.shape
    dq_dtype = dq_dtype or X.dtype
    dev = X.device
    Xq = torch.empty((T, Cw), dtype=dq_dtype, device=dev)
    quant = (bits & ~ACT_SYM) < 16
    cd = torch.empty((T, Cw), dtype=torch.uint8, device=dev) if (codes and quant) else None
    h = torch.empty(T, dtype=torch.float32, device=dev) if (hz and quant) else None
    z = torch.empty(T, dtype=torch.float32, device=dev) if (hz and quant) else None
    _check(lib().oq_act_fakequant_fwd(_ptr(X), _dt(X), T, Cw, bits, _ptr(_f32(s, "s")),
                                      _ptr(_f32(delta, "delta")), _ptr(Xq), _dt(Xq), _ptr(cd),
                                      _ptr(h), _ptr(z), _stream(stream)))
    return Xq, cd, h, z


def act_fakequant_bwd(X, bits, dX_dq, s=None, delta=None, want_dX_tilde=True, stream=None):
    """Returns (dX_tilde | None, d_s, d_delta) (input-path parts of the LET gradients)."""
    T, Cw = X.shape
    dev = X.device
    dxt = torch.empty((T, Cw), dtype=torch.float32, device=dev) if want_dX_tilde else None
    ds = torch.empty(Cw, dtype=torch.float32, device=dev)
    dd = torch.empty(Cw, dtype=torch.float32, device=dev)
    n = C.c_size_t(0)
    _check(lib().oq_act_fakequant_bwd_workspace_size(T, Cw, C.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=dev)
    _check(lib().oq_act_fakequant_bwd(_ptr(X), _dt(X), T, Cw, bits, _ptr(s), _ptr(delta),
                                      _ptr(_f32(dX_dq, "dX_dq")), _ptr(dxt), _ptr(ds), _ptr(dd),
                                      _ptr(ws), n.value, _stream(stream)))
    return dxt, ds, dd


def act_fakequant_bwd_noalloc_into(X, bits, dX_dq, dX_tilde, d_s, d_delta, s=None, delta=None,
                                   stream=None):
    """oq_act_fakequant_bwd_noalloc into caller-provided outputs (any may be
    None): the column partials live in the library's static device scratch,
    so the call allocates nothing."""
    T, Cw = X.shape
    _check(lib().oq_act_fakequant_bwd_noalloc(_ptr(X), _dt(X), T, Cw, bits, _ptr(s), _ptr(delta),
                                              _ptr(_f32(dX_dq, "dX_dq")), _ptr(dX_tilde),
                                              _ptr(d_s), _ptr(d_delta), _stream(stream)))


def let_absorb(P, s, delta, b=None, stream=None):
    """LET absorbed into the producer of a site's input: P [C] (a norm gain)
    or [C, n] (a previous linear's weight, output channels as rows).
    Returns (P / s row-wise, (b - delta) / s)."""
    Cn = P.shape[0]
    n = P.numel() // Cn if Cn else 0
    P_out = torch.empty_like(P)
    b_out = torch.empty(Cn, dtype=torch.float32, device=P.device)
    _check(lib().oq_let_absorb(_ptr(P), _dt(P), _ptr(b), Cn, n, _ptr(s), _ptr(delta), _ptr(P_out),
                               _ptr(b_out), _stream(stream)))
    return P_out, b_out


def let_init(X, Ws, stream=None):
    """SmoothQuant scale / OS+ shift initialisation.  Returns (s, delta)."""
    T, Cw = X.shape
    dev = X.device
    s = torch.empty(Cw, dtype=torch.float32, device=dev)
    d = torch.empty(Cw, dtype=torch.float32, device=dev)
    ptrs = (C.c_void_p * len(Ws))(*[W.data_ptr() for W in Ws])
    couts = (C.c_int64 * len(Ws))(*[int(W.shape[0]) for W in Ws])
    n = C.c_size_t(0)
    _check(lib().oq_let_init_workspace_size(T, Cw, couts, len(Ws), C.byref(n)))
    ws = torch.empty(n.value, dtype=torch.uint8, device=dev)
    _check(lib().oq_let_init(_ptr(X), _dt(X), T, Cw, ptrs, couts, len(Ws), _dt(Ws[0]), _ptr(s),
                             _ptr(d), _ptr(ws), ws.numel(), _stream(stream)))
    return s, d


def pack_codes(codes, bits, stream=None):
    """Row-wise low-bit strings of integer codes ([c_out, c_in] uint8).
    Returns packed uint8 [c_out, c_in * bits // 8]."""
    if codes.dtype != torch.uint8:
        raise OQError("codes must be uint8")
    c_out, c_in = codes.shape
    packed = torch.empty((c_out, c_in * bits // 8), dtype=torch.uint8, device=codes.device)
    _check(lib().oq_pack_codes(_ptr(codes), c_out, c_in, bits, _ptr(packed), _stream(stream)))
    return packed


def packed_linear(X, packed, bits, group, h, z, B=None, out_dtype=torch.float32, stream=None):
    """Y = X W^T + B with W the dequantised weight of packed codes ([n_tok, c_out])."""
    n_tok, c_in = X.shape
    c_out = packed.shape[0]
    if packed.dtype != torch.uint8 or packed.shape[1] * 8 != c_in * bits:
        raise OQError("packed must be uint8 [c_out, c_in * bits / 8]")
    Y = torch.empty((n_tok, c_out), dtype=out_dtype, device=X.device)
    _check(lib().oq_packed_linear(_ptr(X), _dt(X), n_tok, c_in, _ptr(packed), bits, group,
                                  _ptr(_f32(h, "h")), _ptr(_f32(z, "z")), _ptr(_f32(B, "B")),
                                  c_out, _ptr(Y), _dt(Y), _stream(stream)))
    return Y


def packed_linear_into(X, packed, bits, group, h, z, Y, B=None, stream=None):
    """:func:`packed_linear` writing into an existing ``Y`` [n_tok, c_out]."""
    n_tok, c_in = X.shape
    _check(lib().oq_packed_linear(_ptr(X), _dt(X), n_tok, c_in, _ptr(packed), bits, group,
                                  _ptr(_f32(h, "h")), _ptr(_f32(z, "z")), _ptr(_f32(B, "B")),
                                  packed.shape[0], _ptr(Y), _dt(Y), _stream(stream)))
    return Y


def fp_target(X, W, B=None, stream=None):
    """Channel-major full-precision target Y_T = W X^T + B, [c_out, T]."""
    T, c_in = X.shape
    c_out = W.shape[0]
    if X.dtype != W.dtype:
        raise OQError("X and W must share a dtype")
    Y = torch.empty((c_out, T), dtype=X.dtype, device=X.device)
    _check(lib().oq_fp_target(_ptr(X), _ptr(W), _dt(X), _ptr(_f32(B, "B")), T, c_in, c_out,
                              _ptr(Y), _stream(stream)))
    return Y


def matmul_nt(A, B, out_dtype=torch.float32, stream=None):
    """C = A B^T with A [M, K], B [N, K]."""
    M, K = A.shape
    N = B.shape[0]
    out = torch.empty((M, N), dtype=out_dtype, device=A.device)
    _check(lib().oq_matmul_nt(_ptr(A), _ptr(B), _dt(A), M, N, K, _ptr(out),
                              OQ_BF16 if out_dtype == torch.bfloat16 else OQ_F32, _stream(stream)))
    return out


def matmul(A, B, a_mn=False, b_mn=False, stream=None):
    """fp32 C = opA opB^T of bf16 operands, opA = A [M, K] or (a_mn) A^T with A
    stored [K, M]; opB = B [N, K] or (b_mn) B^T with B stored [K, N]."""
    M = A.shape[1] if a_mn else A.shape[0]
    K = A.shape[0] if a_mn else A.shape[1]
    N = B.shape[1] if b_mn else B.shape[0]
    if (B.shape[0] if b_mn else B.shape[1]) != K:
        raise OQError("inner dimensions differ")
    Cm = torch.empty((M, N), dtype=torch.float32, device=A.device)
    _check(lib().oq_matmul(_ptr(A), int(a_mn), _ptr(B), int(b_mn), M, N, K, _ptr(Cm),
                           _stream(stream)))
    return Cm


def adamw_step(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0, stream=None):
    """In-place AdamW on fp32 tensors p, m, v with gradient g."""
    _check(lib().oq_adamw_step(_ptr(p), _ptr(g), _ptr(m), _ptr(v), p.numel(), lr, beta1, beta2,
                               eps, wd, step, _stream(stream)))


# ------------------------------------------------------------------ block step
class Block:
    """One block's calibration problem: description, parameters, gradient
    buffers, AdamW state and workspace, all device tensors owned by torch.

    ``sites``   list of (width, let, act_bits); act_bits may carry ACT_SYM
    ``linears`` list of (site, c_out, bits, group[, quantizer]); linears of a
                site consecutive; quantizer WQ_LWC (default), WQ_PACT or WQ_LSQ
                (the gamma/beta tensors then hold that quantizer's parameters)
    """

    def __init__(self, T, sites, linears, dtype=torch.bfloat16, device="cuda"):
        self.T, self.sites, self.linears = T, list(sites), list(linears)
        self.dtype, self.device = dtype, device
        d = BlockDesc()
        d.tokens = T
        d.n_sites, d.n_linears = len(sites), len(linears)
        d.dtype = OQ_BF16 if dtype == torch.bfloat16 else OQ_F32
        for k, (w, let, ab) in enumerate(sites):
            d.site_width[k], d.site_let[k], d.site_act_bits[k] = w, int(bool(let)), ab
        for l, lin in enumerate(linears):
            k, co, bits, g = lin[:4]
            d.lin_site[l], d.lin_c_out[l], d.lin_bits[l], d.lin_group[l] = k, co, bits, g
            d.lin_quant[l] = lin[4] if len(lin) > 4 else WQ_LWC
        self.desc = d
        n = C.c_size_t(0)
        _check(lib().oq_block_workspace_size(C.byref(d), C.byref(n)))
        self.ws_bytes = n.value
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.d_gamma = [torch.empty((lin[1], sites[lin[0]][0] // lin[3]), **f32) for lin in linears]
        self.d_beta = [torch.empty_like(t) for t in self.d_gamma]
        self.d_s = [torch.empty(w, **f32) if let else None for (w, let, _) in sites]
        self.d_delta = [torch.empty(w, **f32) if let else None for (w, let, _) in sites]
        self.row_loss = [torch.empty(lin[1], **f32) for lin in linears]
        self.loss = torch.empty((), **f32)
        self.opt_state = None
        self.step_count = 0

    PLAN_FIELDS = ("concurrent", "direct", "wgrad_splits", "fwd_splits", "fused_lwc", "wt_copy")

    def plan(self):
        """The step's launch plan per site: a list of dicts of PLAN_FIELDS."""
        n = len(self.PLAN_FIELDS) * len(self.sites)
        buf = (C.c_int * n)()
        _check(lib().oq_block_plan(C.byref(self.desc), buf, n))
        k = len(self.PLAN_FIELDS)
        return [dict(zip(self.PLAN_FIELDS, buf[i * k:(i + 1) * k])) for i in range(len(self.sites))]

    def init_optimizer(self, lr_lwc=5e-3, lr_let=1e-2, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
        f32 = dict(dtype=torch.float32, device=self.device)
        o = BlockOptim()
        self._mv = []
        for l, t in enumerate(self.d_gamma):
            for name in ("m_gamma", "v_gamma", "m_beta", "v_beta"):
                z = torch.zeros_like(t)
                self._mv.append(z)
                getattr(o, name)[l] = z.data_ptr()
        for k, (w, let, _) in enumerate(self.sites):
            if let:
                for name in ("m_s", "v_s", "m_delta", "v_delta"):
                    z = torch.zeros(w, **f32)
                    self._mv.append(z)
                    getattr(o, name)[k] = z.data_ptr()
        o.lr_lwc, o.lr_let, o.beta1, o.beta2, o.eps, o.wd = lr_lwc, lr_let, beta1, beta2, eps, wd
        self.opt_state = o

    def step(self, X_q, Y_fp_T, W, gamma_logit, beta_logit, s=None, delta=None, B=None,
             update=False, frozen=0, stream=None):
        """One calibration step.  Tensors are lists per site (X_q, s, delta) or
        per linear (Y_fp_T, W, logits, B).  With ``update`` the AdamW state of
        :meth:`init_optimizer` updates the logits, s and delta in place."""
        nl, ns = len(self.linears), len(self.sites)
        prm = BlockParams()
        grd = BlockGrads()
        for l in range(nl):
            prm.W[l] = _ptr(W[l]).value
            prm.B[l] = B[l].data_ptr() if (B is not None and B[l] is not None) else None
            prm.gamma_logit[l] = _ptr(gamma_logit[l]).value
            prm.beta_logit[l] = _ptr(beta_logit[l]).value
            grd.d_gamma_logit[l] = self.d_gamma[l].data_ptr()
            grd.d_beta_logit[l] = self.d_beta[l].data_ptr()
            grd.row_loss[l] = self.row_loss[l].data_ptr()
        for k in range(ns):
            if self.sites[k][1]:
                prm.s[k] = _ptr(s[k]).value
                prm.delta[k] = _ptr(delta[k]).value
                grd.d_s[k] = self.d_s[k].data_ptr()
                grd.d_delta[k] = self.d_delta[k].data_ptr()
        yp = (C.c_void_p * nl)(*[_ptr(y).value for y in Y_fp_T])
        xp = (C.c_void_p * ns)(*[_ptr(x).value if x is not None else None for x in X_q])
        opt = None
        if update:
            if self.opt_state is None:
                raise OQError("call init_optimizer() before update=True")
            self.step_count += 1
            self.opt_state.step = self.step_count
            self.opt_state.frozen = frozen
            opt = C.byref(self.opt_state)
        _check(lib().oq_block_calib_step(C.byref(self.desc), yp, xp, C.byref(prm), C.byref(grd),
                                         opt, _ptr(self.loss), _ptr(self.ws), self.ws_bytes,
                                         _stream(stream)))
        return self.loss

    def _param_structs(self, W, gamma_logit, beta_logit, s, delta, B):
        nl, ns = len(self.linears), len(self.sites)
        prm, grd = BlockParams(), BlockGrads()
        for l in range(nl):
            prm.W[l] = _ptr(W[l]).value
            prm.B[l] = B[l].data_ptr() if (B is not None and B[l] is not None) else None
            prm.gamma_logit[l] = _ptr(gamma_logit[l]).value
            prm.beta_logit[l] = _ptr(beta_logit[l]).value
            grd.d_gamma_logit[l] = self.d_gamma[l].data_ptr()
            grd.d_beta_logit[l] = self.d_beta[l].data_ptr()
            grd.row_loss[l] = self.row_loss[l].data_ptr()
        for k in range(ns):
            if self.sites[k][1]:
                prm.s[k] = _ptr(s[k]).value
                prm.delta[k] = _ptr(delta[k]).value
                grd.d_s[k] = self.d_s[k].data_ptr()
                grd.d_delta[k] = self.d_delta[k].data_ptr()
        return prm, grd

    def save_state(self, path, W, gamma_logit, beta_logit, s=None, delta=None, stream=None):
        """Write Theta (and the AdamW state, when initialised) to ``path``."""
        prm, _ = self._param_structs(W, gamma_logit, beta_logit, s, delta, None)
        opt = C.byref(self.opt_state) if self.opt_state is not None else None
        _check(lib().oq_block_state_save(C.byref(self.desc), C.byref(prm), opt, self.step_count,
                                         os.fsencode(path), _stream(stream)))

    def load_state(self, path, W, gamma_logit, beta_logit, s=None, delta=None, stream=None):
        """Restore Theta (and the AdamW state, when initialised) from ``path``
        into the given tensors; the step count continues from the file."""
        prm, _ = self._param_structs(W, gamma_logit, beta_logit, s, delta, None)
        opt = C.byref(self.opt_state) if self.opt_state is not None else None
        done = C.c_int(0)
        _check(lib().oq_block_state_load(C.byref(self.desc), C.byref(prm), opt, C.byref(done),
                                         os.fsencode(path), _stream(stream)))
        self.step_count = done.value

    def export(self, W, gamma_logit, beta_logit, s=None, delta=None, B=None, stream=None):
        """Algorithm 1's quantised block: per linear (packed codes, h, z, B~)."""
        nl = len(self.linears)
        prm, _ = self._param_structs(W, gamma_logit, beta_logit, s, delta, B)
        outs = []
        for l, lin in enumerate(self.linears):
            k, c_out, bits, group = lin[:4]
            c_in = self.sites[k][0]
            f32 = dict(dtype=torch.float32, device=self.device)
            outs.append((torch.empty((c_out, c_in * bits // 8), dtype=torch.uint8, device=self.device),
                         torch.empty((c_out, c_in // group), **f32),
                         torch.empty((c_out, c_in // group), **f32), torch.empty(c_out, **f32)))
        n = C.c_size_t(0)
        _check(lib().oq_block_export_workspace_size(C.byref(self.desc), C.byref(n)))
        ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device=self.device)
        arr = lambda i: (C.c_void_p * nl)(*[o[i].data_ptr() for o in outs])
        _check(lib().oq_block_export(C.byref(self.desc), C.byref(prm), arr(0), arr(1), arr(2), arr(3),
                                     _ptr(ws), n.value, _stream(stream)))
        return outs

    def calibrate(self, X_q_segs, Y_fp_T_segs, W, gamma_logit, beta_logit, epochs, s=None,
                  delta=None, B=None, frozen=0, stream=None):
        """Algorithm 1's loop: ``epochs`` passes over the segments in order,
        AdamW after every step.  ``X_q_segs[g]`` / ``Y_fp_T_segs[g]`` are the
        per-site / per-linear lists of segment g.  Returns the device tensor of
        the epochs * segments step losses.  ``frozen`` (FREEZE_LWC | FREEZE_LET)
        keeps a parameter set and its AdamW state fixed (iterative training)."""
        if self.opt_state is None:
            raise OQError("call init_optimizer() before calibrate()")
        nl, ns, ng = len(self.linears), len(self.sites), len(X_q_segs)
        prm, grd = self._param_structs(W, gamma_logit, beta_logit, s, delta, B)
        yp = (C.c_void_p * (ng * nl))(*[_ptr(y).value for seg in Y_fp_T_segs for y in seg])
        xp = (C.c_void_p * (ng * ns))(*[_ptr(x).value for seg in X_q_segs for x in seg])
        losses = torch.empty(epochs * ng, dtype=torch.float32, device=self.device)
        self.opt_state.step = self.step_count + 1
        self.opt_state.frozen = frozen
        _check(lib().oq_block_calibrate(C.byref(self.desc), ng, epochs, yp, xp, C.byref(prm),
                                        C.byref(grd), C.byref(self.opt_state), _ptr(losses),
                                        _ptr(self.ws), self.ws_bytes, _stream(stream)))
        self.step_count += epochs * ng
        return losses


# ------------------------------------------------------------------ profiling
def profile_enable(on=True):
    _check(lib().oq_profile_enable(int(on)))


def profile_reset():
    _check(lib().oq_profile_reset())


def profile_read():
    """{kind: (launches, total_ms, work)} for every kernel kind."""
    out = {}
    for i, name in enumerate(PROF_KINDS):
        n, ms, w = C.c_int64(0), C.c_double(0), C.c_double(0)
        _check(lib().oq_profile_read(i, C.byref(n), C.byref(ms), C.byref(w)))
        out[name] = (n.value, ms.value, w.value)
    return out


# ------------------------------------------------------------------ whole LLaMA block
_SIGS_LLAMA = {
    "oq_attention_fwd": (_I, [_P, _P, _P, _I64, _I64, _I, _I, _I, _I, _P, _P, _P, _P]),
    "oq_attention_bwd_workspace_size": (_I, [_I64, _I, _I, _PSZ]),
    "oq_attention_bwd": (_I, [_P, _P, _P, _P, _P, _P, _I64, _I64, _I, _I, _I, _I, _P, _P, _P, _P, _SZ,
                              _P]),
    "oq_llama_workspace_size": (_I, [_P, _PSZ]),
    "oq_llama_block_step": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_llama_calibrate": (_I, [_P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "oq_llama_block_forward": (_I, [_P, _P, _P, _I, _P, _P, _SZ, _P]),
}
SIGNATURES.update(_SIGS_LLAMA)
NL = 7


class LlamaDesc(C.Structure):
    _fields_ = [("tokens", C.c_int64), ("seq_len", C.c_int64), ("hidden", C.c_int64),
                ("ffn", C.c_int64), ("heads", C.c_int), ("kv_heads", C.c_int),
                ("norm_eps", C.c_float), ("rope_base", C.c_float), ("w_bits", C.c_int * NL),
                ("w_group", C.c_int64 * NL), ("act_bits", C.c_int), ("let", C.c_int),
                ("softmax_bits", C.c_int)]


class LlamaParams(C.Structure):
    _fields_ = [("W", C.c_void_p * NL), ("norm1", C.c_void_p), ("norm2", C.c_void_p),
                ("gamma_logit", C.c_void_p * NL), ("beta_logit", C.c_void_p * NL),
                ("s", C.c_void_p * 3), ("delta", C.c_void_p * 3), ("s_a", C.c_void_p)]


class LlamaGrads(C.Structure):
    _fields_ = [("d_gamma_logit", C.c_void_p * NL), ("d_beta_logit", C.c_void_p * NL),
                ("d_s", C.c_void_p * 3), ("d_delta", C.c_void_p * 3), ("d_s_a", C.c_void_p)]


class LlamaOptim(C.Structure):
    _fields_ = [("m_gamma", C.c_void_p * NL), ("v_gamma", C.c_void_p * NL),
                ("m_beta", C.c_void_p * NL), ("v_beta", C.c_void_p * NL),
                ("m_s", C.c_void_p * 3), ("v_s", C.c_void_p * 3), ("m_delta", C.c_void_p * 3),
                ("v_delta", C.c_void_p * 3), ("m_s_a", C.c_void_p), ("v_s_a", C.c_void_p),
                ("step", C.c_int), ("lr_lwc", C.c_double), ("lr_let", C.c_double),
                ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
                ("wd", C.c_double)]


def attention_fwd(Q, K, V, S, H, Hkv, softmax_bits=16, stream=None):
    """Causal attention over bf16 Q [T, H d], K, V [T, Hkv d].  Returns
    (O, LSE, pstat); pstat [H, T, 4] (the quantised rows' max / min and their
    indices) only with softmax_bits < 16, else None."""
    T = Q.shape[0]
    d = Q.shape[1] // H
    O = torch.empty((T, H * d), dtype=torch.float32, device=Q.device)
    lse = torch.empty((H, T), dtype=torch.float32, device=Q.device)
    pstat = (torch.empty((H, T, 4), dtype=torch.float32, device=Q.device)
             if softmax_bits < 16 else None)
    _check(lib().oq_attention_fwd(_ptr(Q), _ptr(K), _ptr(V), T, S, H, Hkv, d, softmax_bits,
                                  _ptr(O), _ptr(lse), _ptr(pstat), _stream(stream)))
    return O, lse, pstat


def attention_bwd(Q, K, V, dO, lse, S, H, Hkv, softmax_bits=16, pstat=None, stream=None):
    """Gradients of :func:`attention_fwd` for bf16 dO [T, H d], from its LSE
    (and pstat with softmax_bits < 16).  Returns (dQ, dK, dV) fp32."""
    T = Q.shape[0]
    d = Q.shape[1] // H
    f32 = dict(dtype=torch.float32, device=Q.device)
    dQ = torch.empty((T, H * d), **f32)
    dK = torch.empty((T, Hkv * d), **f32)
    dV = torch.empty((T, Hkv * d), **f32)
    n = C.c_size_t(0)
    _check(lib().oq_attention_bwd_workspace_size(T, H, softmax_bits, C.byref(n)))
    ws = torch.empty(n.value, dtype=torch.uint8, device=Q.device)
    _check(lib().oq_attention_bwd(_ptr(Q), _ptr(K), _ptr(V), _ptr(dO), _ptr(lse), _ptr(pstat), T,
                                  S, H, Hkv, d, softmax_bits, _ptr(dQ), _ptr(dK), _ptr(dV),
                                  _ptr(ws), n.value, _stream(stream)))
    return dQ, dK, dV


class LlamaBlock:
    """One whole LLaMA block's calibration problem (oq_llama_block_step):
    description, gradient buffers, AdamW state and workspace (torch tensors).
    Linears in the order q, k, v, o, gate, up, down."""

    def __init__(self, T, seq_len, hidden, heads, kv_heads, ffn, w_bits, w_group, act_bits=16,
                 let=False, norm_eps=1e-6, rope_base=10000.0, softmax_bits=16, device="cuda"):
        d = LlamaDesc()
        d.tokens, d.seq_len, d.hidden, d.ffn = T, seq_len, hidden, ffn
        d.heads, d.kv_heads = heads, kv_heads
        d.norm_eps, d.rope_base = norm_eps, rope_base
        for l in range(NL):
            d.w_bits[l], d.w_group[l] = w_bits[l], w_group[l]
        d.act_bits, d.let = act_bits, int(bool(let))
        d.softmax_bits = softmax_bits
        self.desc, self.device, self.let = d, device, bool(let)
        self.T, self.D, self.H, self.Hkv, self.F = T, hidden, heads, kv_heads, ffn
        dh = hidden // heads
        self.c_out = [heads * dh, kv_heads * dh, kv_heads * dh, hidden, ffn, ffn, hidden]
        self.c_in = [hidden, hidden, hidden, heads * dh, hidden, hidden, ffn]
        n = C.c_size_t(0)
        _check(lib().oq_llama_workspace_size(C.byref(d), C.byref(n)))
        self.ws_bytes = n.value
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.d_gamma = [torch.empty((co, ci // g), **f32)
                        for co, ci, g in zip(self.c_out, self.c_in, w_group)]
        self.d_beta = [torch.empty_like(t) for t in self.d_gamma]
        site_w = [hidden, heads * dh, hidden]
        self.d_s = [torch.empty(w, **f32) for w in site_w] if let else [None] * 3
        self.d_delta = [torch.empty(w, **f32) for w in site_w] if let else [None] * 3
        self.d_s_a = torch.empty(kv_heads * dh, **f32) if let else None
        self.loss = torch.empty((), **f32)
        self.opt = None
        self.step_count = 0

    def init_optimizer(self, lr_lwc=5e-3, lr_let=1e-2, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
        o = LlamaOptim()
        self._mv = []

        def z(t, name, i=None):
            m = torch.zeros_like(t)
            self._mv.append(m)
            if i is None:
                setattr(o, name, m.data_ptr())
            else:
                getattr(o, name)[i] = m.data_ptr()
        for l in range(NL):
            for nm in ("m_gamma", "v_gamma", "m_beta", "v_beta"):
                z(self.d_gamma[l], nm, l)
        if self.let:
            for k in range(3):
                for nm in ("m_s", "v_s", "m_delta", "v_delta"):
                    z(self.d_s[k], nm, k)
            z(self.d_s_a, "m_s_a")
            z(self.d_s_a, "v_s_a")
        o.lr_lwc, o.lr_let, o.beta1, o.beta2, o.eps, o.wd = lr_lwc, lr_let, beta1, beta2, eps, wd
        self.opt = o
        self.step_count = 0

    def _params(self, W, norm1, norm2, gl=None, bl=None, s=None, delta=None, s_a=None):
        p = LlamaParams()
        for l in range(NL):
            p.W[l] = _ptr(W[l]).value
            if gl is not None:
                p.gamma_logit[l] = _ptr(gl[l]).value
                p.beta_logit[l] = _ptr(bl[l]).value
        p.norm1, p.norm2 = _ptr(_f32(norm1, "norm1")).value, _ptr(_f32(norm2, "norm2")).value
        if self.let and s is not None:
            for k in range(3):
                p.s[k] = _ptr(s[k]).value
                p.delta[k] = _ptr(delta[k]).value
            p.s_a = _ptr(s_a).value
        return p

    def _grads(self):
        g = LlamaGrads()
        for l in range(NL):
            g.d_gamma_logit[l] = self.d_gamma[l].data_ptr()
            g.d_beta_logit[l] = self.d_beta[l].data_ptr()
        if self.let:
            for k in range(3):
                g.d_s[k] = self.d_s[k].data_ptr()
                g.d_delta[k] = self.d_delta[k].data_ptr()
            g.d_s_a = self.d_s_a.data_ptr()
        return g

    def calibrate(self, h0s, targets, W, norm1, norm2, gl, bl, s=None, delta=None, s_a=None,
                  epochs=1, stream=None):
        """Algorithm 1's loop for this block (oq_llama_calibrate): ``epochs``
        passes over the samples (bf16 [T, D] each, inputs and full-precision
        outputs), one AdamW step per sample, parameters updated in place.
        Returns the losses, fp32 [epochs * len(h0s)]."""
        if self.opt is None:
            raise OQError("call init_optimizer() before calibrate")
        n = len(h0s)
        if len(targets) != n or n == 0:
            raise OQError("one target per sample is needed")
        p = self._params(W, norm1, norm2, gl, bl, s, delta, s_a)
        g = self._grads()
        hp = (C.c_void_p * n)(*[_ptr(x).value for x in h0s])
        tp = (C.c_void_p * n)(*[_ptr(x).value for x in targets])
        losses = torch.empty(epochs * n, dtype=torch.float32, device=self.device)
        self.opt.step = self.step_count + 1
        _check(lib().oq_llama_calibrate(C.byref(self.desc), n, epochs, hp, tp, C.byref(p),
                                        C.byref(g), C.byref(self.opt), _ptr(losses), _ptr(self.ws),
                                        self.ws_bytes, _stream(stream)))
        self.step_count += epochs * n
        return losses

    def step(self, h0, target, W, norm1, norm2, gl, bl, s=None, delta=None, s_a=None,
             update=False, stream=None):
        p = self._params(W, norm1, norm2, gl, bl, s, delta, s_a)
        g = LlamaGrads()
        for l in range(NL):
            g.d_gamma_logit[l] = self.d_gamma[l].data_ptr()
            g.d_beta_logit[l] = self.d_beta[l].data_ptr()
        if self.let:
            for k in range(3):
                g.d_s[k] = self.d_s[k].data_ptr()
                g.d_delta[k] = self.d_delta[k].data_ptr()
            g.d_s_a = self.d_s_a.data_ptr()
        opt = None
        if update:
            if self.opt is None:
                raise OQError("call init_optimizer() before update=True")
            self.step_count += 1
            self.opt.step = self.step_count
            opt = C.byref(self.opt)
        _check(lib().oq_llama_block_step(C.byref(self.desc), _ptr(h0), _ptr(target), C.byref(p),
                                         C.byref(g), opt, _ptr(self.loss), _ptr(self.ws),
                                         self.ws_bytes, _stream(stream)))
        return self.loss

    def forward(self, h0, W, norm1, norm2, gl=None, bl=None, s=None, delta=None, s_a=None,
                quantised=True, stream=None):
        """The block's output (bf16 [T, D]): quantised with the given
        parameters, or the full-precision block (Algorithm 1's propagation)."""
        p = self._params(W, norm1, norm2, gl, bl, s, delta, s_a)
        out = torch.empty((self.T, self.D), dtype=torch.bfloat16, device=self.device)
        _check(lib().oq_llama_block_forward(C.byref(self.desc), _ptr(h0), C.byref(p),
                                            int(bool(quantised)), _ptr(out), _ptr(self.ws),
                                            self.ws_bytes, _stream(stream)))
        return out


def llama_algorithm1(blk, blocks, samples, epochs, lr_lwc=5e-3, lr_let=1e-2, stream=None):
    """Algorithm 1 over a stack of LLaMA blocks of one shape (``blk``'s
    descriptor), one block after another.  ``blocks``: per block a dict of
    device tensors W (7), norm1, norm2, gl, bl and, with LET, s, delta, s_a
    (the trainable ones updated in place); ``samples``: the calibration
    inputs, bf16 [T, D] each (batch size 1).  Block i's targets are its
    full-precision outputs on the full-precision stream; it trains from the
    quantised stream with a fresh AdamW state; then the full-precision
    stream moves on through the block unquantised and the quantised stream
    through the block with its learned parameters.  Returns (the losses of
    each block, the final quantised stream)."""
    x_fp, x_q = list(samples), list(samples)
    losses = []
    for b in blocks:
        W, n1, n2 = b["W"], b["norm1"], b["norm2"]
        let = dict(s=b.get("s"), delta=b.get("delta"), s_a=b.get("s_a"))
        targets = [blk.forward(x, W, n1, n2, quantised=False, stream=stream) for x in x_fp]
        blk.init_optimizer(lr_lwc, lr_let)
        losses.append(blk.calibrate(x_q, targets, W, n1, n2, b["gl"], b["bl"], epochs=epochs,
                                    stream=stream, **let))
        x_q = [blk.forward(x, W, n1, n2, b["gl"], b["bl"], quantised=True, stream=stream, **let)
               for x in x_q]
        x_fp = targets
    return losses, x_q
