"""OCP E4M3 ("fn" variant) codec -- oracle, test infrastructure only.

Format (paper section 2.1.1: E4M3 = 4 exponent bits + 3 mantissa bits, range
about [-448, 448]; the encoding family is ref. [12] of section 3.1):

* byte ``S EEEE MMM``; exponent bias 7;
* E >= 1: value = (-1)^S * 2^(E-7) * (1 + M/8);
* E == 0: value = (-1)^S * M * 2^-9   (subnormals; M == 0 is a signed zero);
* S.1111.111 (0x7F / 0xFF) is NaN; there are no infinities, so the largest
  finite magnitude is 0x7E = 2^8 * 1.75 = 448.

The paper does not state the rounding mode, the overflow behaviour or the
treatment of signed zero; the reading taken here is: round-to-nearest,
ties to the even code (RNE), saturating: any magnitude that rounds above
448 -- including +-inf -- becomes +-448; the sign bit of the input is always
kept (so -0 and negative values that round to zero give 0x80).
NaN input gives 0x7F (outside the quantiser's domain; defined for completeness).
"""
import numpy as np

E4M3_MAX = 448.0
NAN_CODE = 0x7F


def decode_table() -> np.ndarray:
    """All 256 codes -> float64 values, straight from the format definition."""
    out = np.empty(256, dtype=np.float64)
    for c in range(256):
        s = -1.0 if (c >> 7) else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            out[c] = np.nan
        elif e == 0:
            out[c] = s * m * 2.0 ** -9
        else:
            out[c] = s * 2.0 ** (e - 7) * (1.0 + m / 8.0)
    return out


_DECODE = decode_table()


def decode(codes: np.ndarray) -> np.ndarray:
    """uint8 codes -> float64 values."""
    return _DECODE[np.asarray(codes, dtype=np.uint8)]


def encode(v) -> np.ndarray:
    """float32 values -> uint8 E4M3 codes (RNE, saturating, sign kept).

    The magnitude is rounded exactly once, from its float32 value, to the
    nearest point of the E4M3 grid:
      * below 2^-6 the grid is the subnormal one, spacing 2^-9;
      * in the binade [2^e, 2^(e+1)), e = -6..8, the spacing is 2^(e-3).
    Multiplying a float32 by a power of two is exact here, so the scaled
    magnitude below is the exact real number, and ``np.rint`` (round half to
    even) performs the single RNE rounding.
    """
    v = np.asarray(v, dtype=np.float32)
    bits = v.view(np.uint32)
    sign = ((bits >> np.uint32(31)) << np.uint32(7)).astype(np.uint8)
    mag = np.abs(v.astype(np.float64))            # exact widening
    is_nan = np.isnan(mag)
    mag = np.where(is_nan, 0.0, mag)

    code = np.zeros(v.shape, dtype=np.int64)
    sub = mag < 2.0 ** -6
    # subnormal range: n = RNE(mag / 2^-9), n in [0, 8]; n == 8 is 2^-6, whose
    # code 0x08 is the smallest normal, so the two ranges join without a gap.
    code = np.where(sub, np.rint(np.minimum(mag, 1.0) * 2.0 ** 9).astype(np.int64), code)
    # normal range: e = floor(log2(mag)); mantissa steps of 2^(e-3)
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.floor(np.log2(np.where(sub, 1.0, np.minimum(mag, 2.0 ** 20))))
    e = e.astype(np.int64)
    # log2 of an exact power of two is exact in IEEE arithmetic, but guard the
    # binade choice anyway so that 2^e <= mag < 2^(e+1) always holds.
    e = np.where(np.ldexp(1.0, e) > mag, e - 1, e)
    e = np.where(np.ldexp(1.0, e + 1) <= mag, e + 1, e)
    capped = np.where(sub, 8.0, np.minimum(mag, 2.0 ** 20))
    n = np.rint(np.ldexp(capped, 3 - e)).astype(np.int64)  # in [8, 16] below 448
    normal_code = ((e + 7) << 3) + (n - 8)          # n == 16 carries into E
    code = np.where(sub, code, normal_code)
    # saturation: everything that rounds past the largest finite value is 448
    code = np.where(mag >= E4M3_MAX, 0x7E, code)
    code = np.minimum(code, 0x7E).astype(np.uint8)
    code = code | sign
    code = np.where(is_nan, NAN_CODE, code).astype(np.uint8)
    return code


def encode_nearest_bruteforce(x: float) -> int:
    """Encode one value by searching every finite code (a pin for ``encode``).

    Picks the finite E4M3 value nearest to x; on an exact tie the code with an
    even mantissa bit wins; magnitudes beyond 448 saturate; the sign of x is
    kept.  Pure Python and slow: for tiny inputs only.
    """
    x = float(np.float32(x))
    neg = np.signbit(np.float32(x))
    a = abs(x)
    best = None
    for c in range(0x7F):                     # 0x00 .. 0x7E: non-negative finite
        val = float(_DECODE[c])
        d = abs(val - a)
        if best is None or d < best[0] or (d == best[0] and (c & 1) == 0):
            best = (d, c)
    code = best[1]
    if a >= E4M3_MAX:
        code = 0x7E
    return code | (0x80 if neg else 0)
