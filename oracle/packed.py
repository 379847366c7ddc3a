"""Oracle: low-bit weight storage and the weight-only quantised linear used to
deploy the calibrated weights (Sec. 4.5 and Table "tab:speed": WxA16 group-wise
models whose stored weights are the integer codes W_q of Eq.2 plus one step
size h and zero point z per group).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Readings of points the paper leaves open (it names the deployment framework
but not a storage format):
  * each output row's codes are stored as one little-endian bit string: code j
    of the row occupies bits j*bits .. j*bits + bits - 1, and bit k of the
    string is bit (k mod 8) of byte k div 8, so a row of C_in codes takes
    C_in * bits / 8 bytes and rows follow each other;
  * h and z are kept per group exactly as Eq.2 produces them (fp32), and the
    weight a deployed linear uses is Eq.2's dequantisation (W_q - z) * h;
  * the deployed linear is Y = X W^T + B with 16-bit (bf16) activations X,
    as in the calibration forward; the oracle evaluates it in fp64.
"""
import numpy as np


def pack_codes(codes, bits):
    """Row-wise little-endian bit string of ``codes`` ([c_out, c_in], values
    below 2**bits); returns uint8 [c_out, c_in * bits / 8]."""
    codes = np.asarray(codes)
    c_out, c_in = codes.shape
    assert (c_in * bits) % 8 == 0
    assert codes.min(initial=0) >= 0 and codes.max(initial=0) < 2 ** bits
    shifts = np.arange(bits, dtype=np.int64)
    # one entry per bit of the string, in string order
    stream = ((codes.astype(np.int64)[:, :, None] >> shifts) & 1).reshape(c_out, c_in * bits)
    return np.packbits(stream.astype(np.uint8), axis=1, bitorder="little")


def unpack_codes(packed, bits, c_in):
    """Inverse of :func:`pack_codes`: uint8 [c_out, c_in * bits / 8] -> int64
    codes [c_out, c_in]."""
    packed = np.asarray(packed, dtype=np.uint8)
    c_out = packed.shape[0]
    stream = np.unpackbits(packed, axis=1, bitorder="little")[:, :c_in * bits]
    stream = stream.reshape(c_out, c_in, bits).astype(np.int64)
    return (stream << np.arange(bits, dtype=np.int64)).sum(axis=2)


def dequant_weight(codes, h, z, group):
    """Eq.2's dequantisation (W_q - z) * h per group, in fp64: [c_out, c_in]."""
    q = np.asarray(codes, np.float64)
    c_out, c_in = q.shape
    hh = np.repeat(np.asarray(h, np.float64).reshape(c_out, c_in // group), group, axis=1)
    zz = np.repeat(np.asarray(z, np.float64).reshape(c_out, c_in // group), group, axis=1)
    return (q - zz) * hh


def packed_linear(X, packed, bits, group, h, z, bias=None):
    """Y = X W^T (+ B) with W the dequantised weight of a packed row-major
    code matrix; X [n, c_in] (its values as given, usually bf16-representable),
    result fp64 [n, c_out]."""
    X = np.asarray(X, np.float64)
    W = dequant_weight(unpack_codes(packed, bits, X.shape[1]), h, z, group)
    Y = X @ W.T
    if bias is not None:
        Y = Y + np.asarray(bias, np.float64)[None, :]
    return Y
