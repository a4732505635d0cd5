"""The FP8 E4M3 format, from its definition (oracle; test infrastructure only).

OCP 8-bit floating point, E4M3 ("FN") variant: 1 sign bit, 4 exponent bits
with bias 7, 3 mantissa bits; exponent field 0 encodes subnormals
m/8 * 2^-6; the all-ones pattern S.1111.111 is NaN; there are no infinities;
the largest finite value is 1.75 * 2^8 = 448.

The paper's facts about it (section "The FP8 Variant of Ozaki II" and the
"e4m3 layout envelope" paragraph): consecutive integers are exact only on
[-16, 16]; the exactly representable integers are M * 2^e with |M| <= 15 and
magnitude <= 448 (so 18, 20, 22 are exact and 17, 19, 21, 23 are not).
"""
from __future__ import annotations


def decode(byte: int) -> float:
    byte &= 0xFF
    sign = -1.0 if byte & 0x80 else 1.0
    e = (byte >> 3) & 0xF
    m = byte & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


def exact_integers() -> list[int]:
    """The set E of integers exactly representable in E4M3 (both signs)."""
    vals = set()
    for b in range(256):
        v = decode(b)
        if v == v and v == int(v):
            vals.add(int(v))
    return sorted(vals)


_ENC = {}
for _b in range(256):
    _v = _decode = decode(_b)
    if _v == _v and _v == int(_v) and int(_v) not in _ENC:
        if _v == 0 and _b != 0:      # keep +0 (byte 0x00) for zero
            continue
        _ENC[int(_v)] = _b


def encode_int(x: int) -> int:
    """The E4M3 byte that represents the integer x exactly (+0 for 0)."""
    try:
        return _ENC[int(x)]
    except KeyError:
        raise ValueError(f"{x} is not exactly representable in E4M3") from None


def in_E(x: int) -> bool:
    return int(x) in _ENC
