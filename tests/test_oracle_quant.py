"""Pins for the oracle's weight format (quantize, dequantize, packing).

Each check rests on something other than the oracle itself: exhaustive search
over all binary16 patterns, exact round trips on values built on the grid, the
round-to-nearest error bound, and an independent bit-by-bit packer."""
import numpy as np
import pytest

from oracle import quant
from inputs import synth

BITS = quant.SUPPORTED_BITS


def _all_finite_halves():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = h.view(np.float16).astype(np.float64)
    ok = np.isfinite(v)
    return h[ok], v[ok]


def _nearest_half_bruteforce(x, hs, vs):
    """Nearest binary16 by search; ties to the pattern with an even mantissa."""
    d = np.abs(vs - x)
    best = d.min()
    cands = hs[d == best]
    if len(cands) > 1:
        even = [c for c in cands if (int(c) & 1) == 0]
        cands = even if even else cands
        # +0 and -0 are both "nearest" to 0: prefer the sign of x
        if best == 0 and x == 0:
            return np.uint16(0x8000 if np.signbit(x) else 0)
    return np.uint16(cands[0])


def test_f64_to_half_matches_exhaustive_search():
    hs, vs = _all_finite_halves()
    pos = vs > 0
    r = np.random.default_rng(1)
    # random magnitudes over the normal and subnormal range, plus exact midpoints
    xs = list(np.exp(r.uniform(np.log(1e-8), np.log(6e4), 400)))
    sv = np.unique(vs[pos])
    mids = (sv[:-1] + sv[1:]) / 2
    xs += list(r.choice(mids, 200, replace=False))
    for x in xs:
        assert quant.f64_to_half_bits(x) == _nearest_half_bruteforce(x, hs, vs), x


@pytest.mark.parametrize("bits", BITS)
def test_roundtrip_exact_on_grid(bits):
    """Blocks built as d * q with max |q| = qmax quantize back to the same codes and scales."""
    r = np.random.default_rng(bits)
    R, K = 6, 128
    qm = quant.qmax(bits)
    # binary16 normal scales
    d = r.uniform(1e-3, 0.1, size=(R, K // 32)).astype(np.float16)
    q = r.integers(-qm, qm + 1, size=(R, K // 32, 32))
    q[:, :, 0] = np.where(r.random((R, K // 32)) < 0.5, qm, -qm)
    w = (q * d.astype(np.float64)[:, :, None]).astype(np.float32).reshape(R, K)
    assert np.array_equal(w.astype(np.float64).reshape(R, K // 32, 32),
                          q * d.astype(np.float64)[:, :, None])  # exact in float32
    codes, scales = quant.quantize(w, bits)
    assert np.array_equal(scales, d.view(np.uint16))
    assert np.array_equal(codes.reshape(R, K // 32, 32).astype(np.int64) - quant.zero_point(bits), q)
    assert np.array_equal(quant.dequantize(codes, scales, bits), w.astype(np.float64))


@pytest.mark.parametrize("bits", BITS)
def test_rounding_error_bound(bits):
    """|w - w_hat| <= d/2 for every weight inside the representable range."""
    w = synth.normal_weights(16, 256, "pin", bits)
    codes, scales = quant.quantize(w, bits)
    what = quant.dequantize(codes, scales, bits)
    d = np.repeat(quant.half_bits_to_f64(scales), 32, axis=1)
    inside = np.abs(w.astype(np.float64)) <= quant.qmax(bits) * d
    err = np.abs(w.astype(np.float64) - what)
    assert np.all(err[inside] <= d[inside] / 2 * (1 + 1e-12))
    # clamped values land on the extreme code
    q = codes.astype(np.int64) - quant.zero_point(bits)
    assert np.all(np.abs(q) <= quant.qmax(bits))
    assert np.all(np.abs(q[~inside]) == quant.qmax(bits))


def test_scale_is_amax_over_qmax_rounded():
    w = np.zeros((1, 32), np.float32)
    w[0, 5] = -0.07
    codes, scales = quant.quantize(w, 4)
    assert quant.half_bits_to_f64(scales)[0, 0] == np.float64(np.float16(0.07 / 7))
    assert codes[0, 5] == 8 - 7
    assert np.all(np.delete(codes[0], 5) == 8)


@pytest.mark.parametrize("bits", BITS)
def test_all_codes_decode(bits):
    K = max(32, 1 << bits)
    codes = (np.arange(K) % (1 << bits)).astype(np.uint8)[None, :]
    scales = np.full((1, K // 32), np.float16(0.5).view(np.uint16), np.uint16)
    got = quant.dequantize(codes, scales, bits)
    assert np.array_equal(got[0], 0.5 * (codes[0].astype(np.float64) - (1 << (bits - 1))))


def test_zero_block():
    codes, scales = quant.quantize(np.zeros((2, 64), np.float32), 3)
    assert np.all(scales == 0) and np.all(codes == 4)
    assert np.all(quant.dequantize(codes, scales, 3) == 0)


def test_two_bit_is_ternary():
    w = synth.normal_weights(8, 256, "pin", "ternary")
    codes, _ = quant.quantize(w, 2)
    assert set(np.unique(codes.astype(int) - 2)) <= {-1, 0, 1}


def _pack_bitwise(codes, bits):
    """Independent packer: append each code's bits to an integer, LSB first."""
    out = []
    for row in codes:
        acc, nbits, data = 0, 0, bytearray()
        for c in row:
            acc |= int(c) << nbits
            nbits += bits
            while nbits >= 8:
                data.append(acc & 0xFF)
                acc >>= 8
                nbits -= 8
        assert nbits == 0
        out.append(list(data))
    return np.array(out, np.uint8)


@pytest.mark.parametrize("bits", BITS)
def test_pack_matches_bitwise_writer_and_roundtrips(bits):
    r = np.random.default_rng(10 + bits)
    codes = r.integers(0, 1 << bits, size=(3, 96)).astype(np.uint8)
    packed = quant.pack(codes, bits)
    assert packed.shape == (3, 96 * bits // 8)
    assert np.array_equal(packed, _pack_bitwise(codes, bits))
    assert np.array_equal(quant.unpack(packed, bits, 96), codes)


def test_pack_three_bit_worked_example():
    """Codes 5, 3, 7, 0, 1 ... : 5 = 101b at bits 0-2, 3 = 011b at 3-5, 7 = 111b at 6-8."""
    codes = np.zeros((1, 32), np.uint8)
    codes[0, :5] = [5, 3, 7, 0, 1]
    packed = quant.pack(codes, 3)
    # bits 0..15: 1,0,1, 1,1,0, 1,1,1, 0,0,0, 1,0,0, 0
    assert packed[0, 0] == 0b11011101
    assert packed[0, 1] == 0b00010001
    assert np.all(packed[0, 2:] == 0)


def test_tensor_bytes_v3():
    # gate/up [2048 x 7168] at 3 bits, down [7168 x 2048] at 4 bits
    assert quant.tensor_bytes(2048, 7168, 3) == 6_422_528
    assert quant.tensor_bytes(7168, 2048, 4) == 8_257_536


def test_dequantize_half_exact_when_representable():
    """d a power of two: every d * (c - z) has at most 8 significant bits, so
    its binary16 rounding is the value itself (closed form)."""
    for bits in BITS:
        z = quant.zero_point(bits)
        codes = np.arange(1 << bits, dtype=np.uint8)
        codes = np.resize(codes, 64).reshape(2, 32)
        scales = np.array([[0x2000], [0x3C00]], np.uint16)     # 2^-7 and 1.0
        got = quant.dequantize_half(codes, scales, bits).view(np.float16).astype(np.float64)
        want = (codes.astype(np.float64) - z) * np.array([[2.0 ** -7], [1.0]])
        assert np.array_equal(got, want), bits


def test_dequantize_half_rounds_worked_example():
    """d = 1 + 2^-10 (0x3C01): 7 d = 7 + 7 * 2^-10 needs 13 bits; binary16 keeps
    11 (spacing 2^-8 in [4, 8)), and 7 * 2^-10 = 1.75 * 2^-8 rounds up to
    2^-7, so 7d -> 7 + 2^-7 (0x4702).  -3 d = -(3 + 3 * 2^-10): spacing 2^-9 in
    [2, 4), 3 * 2^-10 = 1.5 * 2^-9 is a tie between 2^-9 and 2^-8 -> even
    mantissa 2^-8: -(3 + 2^-8) = 0xC202.  d (c - z) with c = z: +0 or -0."""
    codes = np.full((1, 32), 8, np.uint8)
    codes[0, 0] = 15          # c - z = 7
    codes[0, 1] = 5           # c - z = -3
    scales = np.array([[0x3C01]], np.uint16)
    got = quant.dequantize_half(codes, scales, 4)
    assert got[0, 0] == 0x4702
    assert got[0, 1] == 0xC202
    assert np.all(got[0, 2:].view(np.float16) == 0)
