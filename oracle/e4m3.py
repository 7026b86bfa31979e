"""OCP FP8 E4M3 ("e4m3fn") codec, from the format definition (test oracle).

The paper quantizes to e4m3fn, range [-448, 448] (Sec. 3, the paragraph
introducing Eq. (2); format of Micikevicius et al. 2022).  The definition:

* bit 7 sign, bits 6..3 exponent field E (bias 7), bits 2..0 mantissa m;
* E = 0: subnormal, value m * 2^-9 (so 0x00 = +0, 0x80 = -0);
* 1 <= E <= 15: normal, value (1 + m/8) * 2^(E-7);
* E = 15, m = 7 (0x7F / 0xFF) is NaN; there is no infinity, so the largest
  finite magnitude is 0x7E = 1.75 * 2^8 = 448.

``encode_rne`` returns the code of the representable value nearest to y,
ties to the code with an even mantissa (round-to-nearest-even); the paper's
"rounds to the nearest representable value" (Eq. (2)) fixes the nearest
value but not the tie, and ties-to-even is the reading taken here.
"""
import numpy as np

MAX_FINITE = 448.0
NAN_CODES = (0x7F, 0xFF)


def _decode_codes(c):
    """The definition above, applied to int64 codes."""
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return sign * mag


# the value of every code, so that decoding an array is a lookup (same values)
_VALUES = _decode_codes(np.arange(256, dtype=np.int64))


def decode(codes):
    """Value (float64) of each e4m3fn code; NaN for 0x7F / 0xFF."""
    return _VALUES[np.asarray(codes, dtype=np.uint8)]


def _encode_block(y):
    """encode_rne on a float64 array (no checks)."""
    a = np.abs(y)
    code = np.zeros(a.shape, dtype=np.int64)

    sub = a < 2.0 ** -6
    # subnormal binade: multiples of 2^-9; rint() is round-half-even
    code[sub] = np.rint(a[sub] * 2.0 ** 9).astype(np.int64)  # 8 -> 0x08 = 2^-6

    nrm = ~sub
    _, ex = np.frexp(a[nrm])            # a = f * 2^ex, f in [0.5, 1)
    e = ex - 1                          # a in [2^e, 2^(e+1))
    q = np.rint(np.ldexp(a[nrm], 3 - e)).astype(np.int64)  # in [8, 16]
    carry = q == 16
    e = np.where(carry, e + 1, e)
    q = np.where(carry, 8, q)
    code[nrm] = ((e + 7) << 3) | (q - 8)

    code = code | np.where(np.signbit(y), 0x80, 0)
    return code.astype(np.uint8)


def encode_rne(y):
    """e4m3fn code (uint8) of each finite y with |y| <= 448, nearest-even.

    y may be float32 or float64; it is widened to float64 exactly.  For a
    normal target the magnitude is written a = 2^e * q / 8 with q in [8, 16);
    q is rounded half-to-even to an integer (a power-of-two scaling, so the
    rounding is of y itself), and a carry to 16 moves to the next binade.
    Below 2^-6 the spacing is the subnormal step 2^-9.  Each element is coded
    on its own; large arrays go through in pieces of 2^18 elements only to keep
    the temporaries small.
    """
    y = np.asarray(y)
    flat = y.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint8)
    piece = 1 << 18
    for i in range(0, flat.size, piece):
        yi = flat[i:i + piece].astype(np.float64)
        if not np.all(np.abs(yi) <= MAX_FINITE):   # also false for NaN
            raise ValueError("encode_rne needs finite inputs with |y| <= 448")
        out[i:i + piece] = _encode_block(yi)
    return out.reshape(y.shape)


def round_to_e4m3(y):
    """The value nearest to y in e4m3fn (float64), via encode then decode."""
    return decode(encode_rne(y))
