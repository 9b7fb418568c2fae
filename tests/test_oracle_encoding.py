"""Pins for oracle.encoding against the mathematics, not against itself.

* exhaustive over all 2^16 words: exact refinement, zero-filled low byte;
* the value of every BASE word against an independent closed form built
  from ``math.frexp`` (no bit operations): for bf16 the low byte holds the
  exponent's least significant bit plus the 7 mantissa bits, so BASE rounds
  the magnitude down to an even power of two's exponent; for fp16 it keeps
  2 mantissa bits, i.e. truncation toward zero to 2^(E-2);
* hand-worked words from ``tests/golden/base_encoding.txt``.
"""

import math
import os

import numpy as np
import pytest

from oracle import encoding

ALL = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)


def test_refinement_is_exact_for_every_word():
    hi = encoding.hi_byte(ALL)
    lo = encoding.lo_byte(ALL)
    assert np.array_equal(encoding.refine_word(hi, lo), ALL)
    # the two bytes are the two halves of the word, nothing else
    assert np.array_equal(hi.astype(np.int64) * 256 + lo.astype(np.int64), ALL.astype(np.int64))


def test_base_word_zero_fills_low_byte():
    b = encoding.base_word(encoding.hi_byte(ALL))
    assert np.array_equal(b.astype(np.int64), (ALL.astype(np.int64) // 256) * 256)


def _bf16_value_by_fields(w):
    sign = -1.0 if w >> 15 else 1.0
    e = (w >> 7) & 0xFF
    m = w & 0x7F
    if e == 0:
        return sign * m * 2.0 ** -133
    if e == 255:
        return math.nan if m else sign * math.inf
    return sign * (1 + m / 128) * 2.0 ** (e - 127)


def _bf16_base_closed_form(x):
    """sign(x) * 2^(2*floor(e/2) - 127) with e the biased exponent, or 0."""
    if x == 0 or (math.isfinite(x) and abs(x) < 2.0 ** -126):
        return math.copysign(0.0, x)
    if not math.isfinite(x):
        return math.copysign(2.0 ** 127, x) if not math.isnan(x) else None
    _, e2 = math.frexp(abs(x))          # |x| = f * 2^e2, f in [0.5, 1)
    biased = (e2 - 1) + 127
    even = biased - (biased % 2)
    return math.copysign(2.0 ** (even - 127), x) if even > 0 else math.copysign(0.0, x)


def test_bf16_base_value_matches_closed_form_for_every_word():
    vals = encoding.words_to_f64(ALL, "bf16")
    base = encoding.base_value(ALL, "bf16")
    for w in range(1 << 16):
        x = vals[w]
        assert (x == _bf16_value_by_fields(w)) or (math.isnan(x) and math.isnan(_bf16_value_by_fields(w)))
        expect = _bf16_base_closed_form(x)
        if expect is None:       # NaN: high byte of a NaN is 0x7F / 0xFF -> +-2^127
            assert abs(base[w]) == 2.0 ** 127
            continue
        assert base[w] == expect and math.copysign(1, base[w]) == math.copysign(1, expect), hex(w)


def _fp16_base_closed_form(x):
    """Truncation toward zero to 2 mantissa bits: ulp = 2^(max(E,-14) - 2)."""
    if not math.isfinite(x):
        return None
    if x == 0:
        return x
    _, e2 = math.frexp(abs(x))
    exp = max(e2 - 1, -14)
    ulp = 2.0 ** (exp - 2)
    return math.copysign(math.floor(abs(x) / ulp) * ulp, x)


def test_fp16_base_value_matches_closed_form_for_every_finite_word():
    vals = encoding.words_to_f64(ALL, "fp16")
    base = encoding.base_value(ALL, "fp16")
    for w in range(1 << 16):
        expect = _fp16_base_closed_form(vals[w])
        if expect is None:
            continue
        assert base[w] == expect and math.copysign(1, base[w]) == math.copysign(1, expect), hex(w)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_base_never_grows_and_keeps_sign(dtype):
    x = encoding.words_to_f64(ALL, dtype)
    b = encoding.base_value(ALL, dtype)
    fin = np.isfinite(x)
    assert np.all(np.abs(b[fin]) <= np.abs(x[fin]))
    assert np.all(np.signbit(b[fin]) == np.signbit(x[fin]))
    nz = fin & (b != 0)
    ratio = b[nz] / x[nz]
    lo_bound = 0.25 if dtype == "bf16" else 0.5      # worst case 1 - 2^-? truncation
    assert ratio.min() > lo_bound and ratio.max() <= 1.0


def test_golden_words(golden_dir):
    path = os.path.join(golden_dir, "base_encoding.txt")
    n = 0
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        dtype, w, bw, lo, val = line.split()
        w, bw, lo, val = int(w, 16), int(bw, 16), int(lo, 16), float(val)
        word = np.array([w], dtype=np.uint16)
        assert int(encoding.base_word(encoding.hi_byte(word))[0]) == bw
        assert int(encoding.lo_byte(word)[0]) == lo
        assert float(encoding.base_value(word, dtype)[0]) == val
        assert int(encoding.refine_word(encoding.hi_byte(word), encoding.lo_byte(word))[0]) == w
        n += 1
    assert n >= 12
