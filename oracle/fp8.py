"""fp8 (OCP E4M3FN) KV codes (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Storing K and V pages as 8-bit codes halves the bytes a decode step streams
per cached token.  That traffic bounds long-context decode (Introduction;
Background, "Hardware-Workload Interaction").  The format is the OCP
8-bit E4M3 "FN" encoding:
* sign bit, 4 exponent bits (bias 7), 3 mantissa bits;
* subnormals m * 2^-9;
* largest finite value 448;
* no infinities; S.1111.111 is NaN.

A value x is stored as code(x / scale), rounding to nearest with ties to
even, saturating at +-448 and keeping the sign (also of values that round to
zero); it reads back as value(code) * scale.
"""

from __future__ import annotations

import numpy as np

MAX_E4M3 = 448.0


def e4m3_values() -> np.ndarray:
    """float64 value of each of the 256 codes (NaN for the two NaN codes)."""
    out = np.empty(256, dtype=np.float64)
    for c in range(256):
        sign = -1.0 if c & 0x80 else 1.0
        e, m = (c >> 3) & 0xF, c & 0x7
        if e == 0xF and m == 0x7:
            out[c] = np.nan
        elif e == 0:
            out[c] = sign * m * 2.0 ** -9
        else:
            out[c] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_VALUES = e4m3_values()
# finite non-negative codes in increasing value order: 0x00 .. 0x7E
_POS = _VALUES[:0x7F]


def e4m3_encode(x) -> np.ndarray:
    """Nearest code (ties to the even code) of each float, saturating at 448."""
    a = np.asarray(x, dtype=np.float64)
    mag = np.minimum(np.abs(a), MAX_E4M3)
    hi = np.clip(np.searchsorted(_POS, mag, side="left"), 0, 0x7E)  # first value >= mag
    lo = np.maximum(hi - 1, 0)
    d_lo, d_hi = mag - _POS[lo], _POS[hi] - mag
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    code = np.where(mag == _POS[hi], hi, code).astype(np.uint8)  # exact values
    neg = np.signbit(a)  # the sign is kept, also on values that round to zero
    return (code | (neg.astype(np.uint8) << 7)).astype(np.uint8)


def e4m3_decode(codes) -> np.ndarray:
    return _VALUES[np.asarray(codes, dtype=np.uint8)]


def quantize_dequantize(x, scale: float) -> np.ndarray:
    """What a page stores for x and reads back: value(code(x / scale)) * scale."""
    return e4m3_decode(e4m3_encode(np.asarray(x, dtype=np.float64) / scale)) * scale


def paged_decode_attention_fp8(q, k_codes, v_codes, k_scale: float, v_scale: float,
                               block_table, lens) -> np.ndarray:
    """Paged decode attention over e4m3 K/V code pools ``[P, Hkv, 16, Dh]``:
    the codes are read back as value(code) * scale and the plain attention
    definition applies."""
    from .paged import paged_decode_attention
    return paged_decode_attention(q, e4m3_decode(k_codes) * k_scale,
                                  e4m3_decode(v_codes) * v_scale, block_table, lens)
