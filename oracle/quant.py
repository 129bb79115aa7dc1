"""Oracle: the block-quantized weight format.  TEST INFRASTRUCTURE ONLY.

Section 3.3 of the paper quantizes the pruned model to a low base precision and
then gives each tensor its own bit width under a memory budget.  The paper's
formats are llama.cpp's; this library uses a plain symmetric block format
instead, and this module is its definition:

* a tensor is a row-major matrix ``[R, K]`` with ``K % 32 == 0``;
* every run of 32 consecutive weights in a row (a *block*) has one scale
  ``d``, stored as an IEEE binary16 bit pattern;
* every weight has a ``b``-bit unsigned code ``c`` (``b`` in 2, 3, 4 and,
  for the wider widths, 5, 6, 8), and its value is ``d * (c - 2**(b-1))``.
  All ``2**b`` codes are valid when decoding;
* packing: the 32 codes of a block form one little-endian bit string of
  ``32*b`` bits (``4*b`` bytes): code ``i`` occupies bits ``[i*b, i*b + b)``.
  Blocks follow each other along the row; scales live in a separate array.

The quantizer (round to nearest, ties to even, symmetric range ``+-qmax`` with
``qmax = 2**(b-1) - 1``) only makes test inputs: the library never quantizes
on the forward path.
"""
import numpy as np

BLOCK = 32
SUPPORTED_BITS = (2, 3, 4, 5, 6, 8)


def zero_point(bits):
    """Code that decodes to 0: ``2**(bits-1)``."""
    return 1 << (bits - 1)


def qmax(bits):
    """Largest magnitude the symmetric quantizer emits: ``2**(bits-1) - 1``."""
    return (1 << (bits - 1)) - 1


def half_bits_to_f64(h):
    """binary16 bit patterns (uint16) -> float64, exactly."""
    return np.asarray(h, dtype=np.uint16).view(np.float16).astype(np.float64)


def f64_to_half_bits(v):
    """float64 -> nearest binary16 (ties to even), as uint16 bit patterns.

    numpy converts double to half directly (no detour through float32), which
    the tests check against an exhaustive search over all 65536 patterns."""
    return np.asarray(v, dtype=np.float64).astype(np.float16).view(np.uint16)


def quantize(w, bits):
    """Quantize float32 ``w[R, K]`` -> (codes uint8 ``[R, K]``, scales uint16 ``[R, K/32]``).

    Per block: ``amax = max |w|``; ``d = half(amax / qmax)`` (quotient in
    float64, one rounding to binary16); if ``d == 0`` every code is the zero
    point; else ``q = clamp(rint(w / d), -qmax, qmax)`` computed in float64
    with the already-rounded ``d``; ``c = q + 2**(b-1)``.
    """
    w = np.asarray(w, dtype=np.float32)
    R, K = w.shape
    assert K % BLOCK == 0 and bits in SUPPORTED_BITS
    nb = K // BLOCK
    wb = w.reshape(R, nb, BLOCK).astype(np.float64)
    amax = np.abs(wb).max(axis=2)
    scales = f64_to_half_bits(amax / qmax(bits))
    d = half_bits_to_f64(scales)[:, :, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(d > 0, np.rint(wb / np.where(d > 0, d, 1.0)), 0.0)
    q = np.clip(q, -qmax(bits), qmax(bits))
    codes = (q + zero_point(bits)).astype(np.uint8).reshape(R, K)
    return codes, scales


def dequantize(codes, scales, bits):
    """codes ``[R, K]`` + scales ``[R, K/32]`` -> float64 ``[R, K]``.

    ``d * (c - 2**(b-1))``: the product of a binary16 value and an integer of
    at most 8 bits is exact in float32, so this float64 result is also the
    exact float32 weight."""
    codes = np.asarray(codes)
    R, K = codes.shape
    q = codes.astype(np.float64) - zero_point(bits)
    d = half_bits_to_f64(scales)
    return (q.reshape(R, K // BLOCK, BLOCK) * d[:, :, None]).reshape(R, K)


def dequantize_half(codes, scales, bits):
    """The weights rounded once to binary16: ``half(d * (c - 2**(b-1)))`` as
    uint16 bit patterns ``[R, K]`` (round to nearest, ties to even, from the
    exact value).  This is what a binary16 matrix product sees of the
    format's weights."""
    return f64_to_half_bits(dequantize(codes, scales, bits))


def pack(codes, bits):
    """codes ``[R, K]`` (each < 2**bits) -> packed bytes ``[R, K*bits/8]``."""
    codes = np.asarray(codes, dtype=np.uint8)
    R, K = codes.shape
    assert K % BLOCK == 0 and int(codes.max(initial=0)) < (1 << bits)
    # bit j of code i, least significant first, as one little-endian bit string
    shifts = np.arange(bits, dtype=np.uint8)
    bitplanes = (codes[:, :, None] >> shifts) & 1          # [R, K, bits]
    return np.packbits(bitplanes.reshape(R, K * bits), axis=1, bitorder="little")


def unpack(packed, bits, K):
    """packed bytes ``[R, K*bits/8]`` -> codes uint8 ``[R, K]``.

    Bit ``j`` of code ``i`` is bit ``i*bits + j`` of the row's bit string."""
    packed = np.asarray(packed, dtype=np.uint8)
    R = packed.shape[0]
    bitstr = np.unpackbits(packed, axis=1, bitorder="little")[:, : K * bits]
    codes = np.zeros((R, K), np.uint8)
    for j in range(bits):
        codes |= bitstr[:, j::bits] << np.uint8(j)
    return codes


def tensor_bytes(rows, K, bits):
    """Bytes of one tensor in this format: codes plus binary16 scales."""
    return rows * K * bits // 8 + rows * (K // BLOCK) * 2
