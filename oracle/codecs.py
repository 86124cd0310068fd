"""Number-format codecs written from the format definitions (oracle side).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper's generated kernels run the matmul in a 16-bit float format with
fp32 accumulation and fp32 post-processing (§IV-B, mixed-precision
execution). On gfx950 the 16-bit operand format is bfloat16 and the 8-bit one
is OCP FP8 E4M3 ("e4m3fn"). The oracle must see the *exact* values the GPU
consumes, so it decodes the stored bit patterns itself, field by field, and
models the storage roundings the method performs (bf16 RNE, e4m3 RNE with
saturation) from the definitions below, not from a library cast.

bfloat16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits; the upper
half of an IEEE-754 binary32. Normal value (-1)^s · 2^(e-127) · (1 + f/2^7);
subnormal (e = 0) (-1)^s · 2^-126 · f/2^7; e = 255 encodes inf (f = 0) / NaN.

OCP FP8 E4M3 (e4m3fn): 1 sign bit, 4 exponent bits (bias 7), 3 fraction
bits. Normal (-1)^s · 2^(e-7) · (1 + f/8); subnormal (e = 0)
(-1)^s · 2^-6 · f/8. There are no infinities; S.1111.111 is NaN, so the
largest finite magnitude is 1.75 · 2^8 = 448 and the smallest subnormal 2^-9.
"""

import numpy as np

E4M3_MAX = 448.0


def bf16_decode(bits):
    """Decode bf16 bit patterns (uint16 array) to fp64, exactly, from fields."""
    b = np.asarray(bits).astype(np.uint32)
    s = (b >> 15) & 1
    e = ((b >> 7) & 0xFF).astype(np.int64)
    f = (b & 0x7F).astype(np.float64)
    sign = np.where(s == 1, -1.0, 1.0)
    normal = np.ldexp(1.0 + f / 128.0, (e - 127).astype(np.int32))
    sub = np.ldexp(f / 128.0, -126)
    val = np.where(e == 0, sub, normal)
    val = np.where((e == 255) & (f == 0), np.inf, val)
    val = np.where((e == 255) & (f != 0), np.nan, val)
    return sign * val


def _round_to_grid(x, mant_bits, min_exp):
    """Round fp64 x to nearest with ties to even onto the grid of a binary
    format with ``mant_bits`` fraction bits whose smallest normal exponent is
    ``min_exp`` (exponent range above is left unbounded; callers handle
    overflow). Returns fp64 values exactly on that grid."""
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    # |x| in [2^(E), 2^(E+1)) with E = floor(log2|x|); frexp gives x = m·2^p, m in [0.5,1)
    _, p = np.frexp(ax)
    E = p.astype(np.int64) - 1
    E = np.maximum(E, min_exp)                    # subnormal range shares the min_exp ulp
    ulp_exp = (E - mant_bits).astype(np.int32)
    q = np.ldexp(ax, -ulp_exp)                     # exact scaling by a power of two
    q = np.rint(q)                                 # numpy rint = round half to even
    r = np.ldexp(q, ulp_exp)
    r = np.where(ax == 0, 0.0, r)
    return np.copysign(r, x)


def bf16_encode_rne(x):
    """Round fp64 values to bf16 (RNE, IEEE overflow to inf) and return the
    uint16 bit patterns. NaN inputs are not supported (never exercised)."""
    x = np.asarray(x, dtype=np.float64)
    r = _round_to_grid(x, 7, -126)
    # largest finite bf16 is (2 - 2^-7)·2^127; values that rounded past it overflow
    r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, r), r)
    # every r is exactly representable in binary32, whose upper half is the bf16 word
    bits32 = r.astype(np.float32).view(np.uint32)
    return (bits32 >> 16).astype(np.uint16)


def _e4m3_decode_fields(codes):
    """Decode OCP e4m3fn bytes to fp64, exactly, from the fields."""
    c = np.asarray(codes).astype(np.uint32)
    s = (c >> 7) & 1
    e = ((c >> 3) & 0xF).astype(np.int64)
    f = (c & 0x7).astype(np.float64)
    sign = np.where(s == 1, -1.0, 1.0)
    normal = np.ldexp(1.0 + f / 8.0, (e - 7).astype(np.int32))
    sub = np.ldexp(f / 8.0, -6)
    val = np.where(e == 0, sub, normal)
    val = np.where((e == 15) & (f == 7), np.nan, val)
    return sign * val


# the 256 code values, decoded once from the fields
_E4M3_VALUES = _e4m3_decode_fields(np.arange(256))


def e4m3_decode(codes):
    """Decode OCP e4m3fn bytes (uint8 array) to fp64, exactly: the value of
    each code as the field decode above gives it."""
    return _E4M3_VALUES[np.asarray(codes).astype(np.uint8)]


def e4m3_encode_rne_sat(x):
    """Round fp64 values to e4m3fn with round-to-nearest-even and saturation
    to ±448 (no NaN produced for finite input); return uint8 codes."""
    x = np.asarray(x, dtype=np.float64)
    r = _round_to_grid(x, 3, -6)
    r = np.clip(r, -E4M3_MAX, E4M3_MAX)
    ar = np.abs(r)
    _, p = np.frexp(ar)
    E = p.astype(np.int64) - 1
    is_sub = ar < 2.0 ** -6
    e_field = np.where(is_sub, 0, E + 7)
    frac = np.where(is_sub, ar / 2.0 ** -9, (ar / np.ldexp(1.0, E.astype(np.int32)) - 1.0) * 8.0)
    frac = np.where(ar == 0, 0.0, frac)
    e_field = np.where(ar == 0, 0, e_field)
    code = (e_field.astype(np.uint32) << 3) | np.rint(frac).astype(np.uint32)
    code = code | np.where(np.signbit(r), 0x80, 0).astype(np.uint32)
    return code.astype(np.uint8)


def f32_round(x):
    """Round fp64 values to the nearest binary32 (IEEE RNE) and return fp64.

    Used only where the method takes an integer-valued decision (an e4m3
    code) in fp32 and the oracle must take the same decision in the same
    precision."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
