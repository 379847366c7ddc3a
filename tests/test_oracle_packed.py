"""Pins for the oracle's low-bit weight storage and weight-only quantised linear
(Sec. 4.5): a hand-worked bit string, the string read as one integer, the usual
nibble and byte layouts, scalar loops on tiny inputs, closed forms, and a tie
to the Eq.2 quantiser's own dequantised weights."""
import numpy as np
import pytest

from oracle.packed import dequant_weight, pack_codes, packed_linear, unpack_codes
from oracle.quant import minmax_quant_rows


def test_hand_worked_three_bit_row():
    # codes 1..7, 0 at 3 bits each, least significant bit first:
    # 1 + 2*8 + 3*64 + 4*512 + 5*4096 + 6*32768 + 7*262144 = 2054353 = 0x1F58D1
    got = pack_codes(np.array([[1, 2, 3, 4, 5, 6, 7, 0]]), 3)
    assert got.tolist() == [[0xD1, 0x58, 0x1F]]


@pytest.mark.parametrize("bits", [2, 3, 4, 5, 6, 7, 8])
def test_row_string_is_the_little_endian_integer(bits):
    rng = np.random.default_rng(bits)
    codes = rng.integers(0, 2 ** bits, size=(5, 64))
    got = pack_codes(codes, bits)
    assert got.shape == (5, 64 * bits // 8) and got.dtype == np.uint8
    for o in range(codes.shape[0]):
        v = 0
        for j, c in enumerate(codes[o].tolist()):
            v += c << (bits * j)
        assert bytes(got[o]) == v.to_bytes(64 * bits // 8, "little")
    assert np.array_equal(unpack_codes(got, bits, 64), codes)


def test_nibble_and_byte_layouts():
    rng = np.random.default_rng(7)
    c4 = rng.integers(0, 16, size=(3, 32))
    assert np.array_equal(pack_codes(c4, 4), (c4[:, 0::2] | (c4[:, 1::2] << 4)).astype(np.uint8))
    c2 = rng.integers(0, 4, size=(3, 32))
    want = c2[:, 0::4] | (c2[:, 1::4] << 2) | (c2[:, 2::4] << 4) | (c2[:, 3::4] << 6)
    assert np.array_equal(pack_codes(c2, 2), want.astype(np.uint8))
    c8 = rng.integers(0, 256, size=(3, 32))
    assert np.array_equal(pack_codes(c8, 8), c8.astype(np.uint8))


def test_linear_scalar_loops():
    rng = np.random.default_rng(3)
    bits, group, c_in, c_out, n = 3, 4, 8, 3, 2
    q = rng.integers(0, 8, size=(c_out, c_in))
    h = rng.uniform(0.01, 0.1, size=(c_out, c_in // group)).astype(np.float32)
    z = rng.integers(0, 8, size=(c_out, c_in // group)).astype(np.float32)
    X = rng.standard_normal((n, c_in))
    B = rng.standard_normal(c_out)
    got = packed_linear(X, pack_codes(q, bits), bits, group, h, z, B)
    for t in range(n):
        for o in range(c_out):
            acc = float(B[o])
            for c in range(c_in):
                g = c // group
                acc += X[t, c] * (q[o, c] - float(z[o, g])) * float(h[o, g])
            assert got[t, o] == pytest.approx(acc, rel=1e-12, abs=1e-12)


def test_linear_closed_forms():
    rng = np.random.default_rng(5)
    bits, group, c_in, c_out = 4, 32, 64, 6
    q = rng.integers(0, 16, size=(c_out, c_in))
    h = rng.uniform(0.01, 0.1, size=(c_out, 2)).astype(np.float32)
    z = rng.integers(0, 16, size=(c_out, 2)).astype(np.float32)
    P = pack_codes(q, bits)
    # a one-hot token reads one column of the dequantised weight exactly
    for c in (0, 31, 32, 63):
        x = np.zeros((1, c_in))
        x[0, c] = 1.0
        col = (q[:, c] - z[:, c // group].astype(np.float64)) * h[:, c // group].astype(np.float64)
        assert np.array_equal(packed_linear(x, P, bits, group, h, z)[0], col)
    # codes equal to the zero point dequantise to 0: the output is the bias
    zq = np.repeat(z.astype(np.int64), group, axis=1)
    B = rng.standard_normal(c_out)
    Y = packed_linear(rng.standard_normal((3, c_in)), pack_codes(zq, bits), bits, group, h, z, B)
    assert np.array_equal(Y, np.broadcast_to(B, Y.shape))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_linear_matches_eq2_dequantised_weight(bits):
    # codes, h and z from the Eq.2 quantiser (gamma = beta = 1) of a random
    # weight: the packed linear uses exactly that quantiser's dequantised weight
    rng = np.random.default_rng(11 + bits)
    c_out, c_in, group = 8, 256, 64
    W = (0.02 * rng.standard_normal((c_out, c_in))).astype(np.float32)
    st = minmax_quant_rows(W.reshape(-1, group), np.ones(c_out * c_in // group, np.float32),
                           np.ones(c_out * c_in // group, np.float32), bits)
    q = st["q"].reshape(c_out, c_in).astype(np.int64)
    h = st["h"].reshape(c_out, c_in // group)
    z = st["z"].reshape(c_out, c_in // group)
    wdq = st["wdq"].reshape(c_out, c_in).astype(np.float64)
    assert np.allclose(dequant_weight(q, h, z, group), wdq, rtol=1e-6, atol=0)
    X = rng.standard_normal((4, c_in))
    Y = packed_linear(X, pack_codes(q, bits), bits, group, h, z)
    ref = X @ wdq.T
    # the two weights differ by fp32 rounding of (q - z) * h only
    assert np.all(np.abs(Y - ref) <= 1e-6 * (np.abs(X) @ np.abs(wdq).T))
