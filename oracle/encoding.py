"""TARGET / BASE / refinement encoding of one 16-bit KV word (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definitions (§3, opening paragraph; App. B.2 "Transition Protocols";
§3.2 and App. B.3 for how BASE is executed):

* TARGET is the native 16-bit representation of a K or V element.
* BASE keeps the high-order 8 bits of that word.  Nothing is rounded: the
  low byte is simply dropped.  Rounding would make exact refinement from the
  stored low byte impossible, so truncation is the only reading compatible
  with "refine exactly".
* The remaining low-order 8 bits are the refinement bits; putting them back
  under the high byte restores TARGET bit for bit, with no scale and no
  dequantization transform.
* To execute on BASE, the stored byte is put back in the high-order position
  of a 16-bit word and the low byte is zero-filled; the result is read in
  the native datatype.

Everything here works on raw unsigned integer words with bit operations only,
never on float arithmetic, so special values (signed zeros, subnormals,
infinities, NaNs) follow the definition exactly.
"""

import numpy as np

DTYPES = ("bf16", "fp16")


def hi_byte(words):
    """BASE byte of each 16-bit TARGET word: bits 15..8 (§3; App. B.2)."""
    w = np.asarray(words, dtype=np.uint16)
    return (w >> np.uint16(8)).astype(np.uint8)


def lo_byte(words):
    """Refinement byte of each TARGET word: bits 7..0 (§3; App. B.2)."""
    w = np.asarray(words, dtype=np.uint16)
    return (w & np.uint16(0xFF)).astype(np.uint8)


def base_word(hi):
    """16-bit word executed for a BASE byte: byte in the high position, zero low
    byte (§3.2; App. B.3)."""
    h = np.asarray(hi, dtype=np.uint8)
    return (h.astype(np.uint16) << np.uint16(8)).astype(np.uint16)


def refine_word(hi, lo):
    """Exact TARGET word restored from its BASE byte and refinement byte
    (§3; App. B.2)."""
    h = np.asarray(hi, dtype=np.uint8).astype(np.uint16)
    l = np.asarray(lo, dtype=np.uint8).astype(np.uint16)
    return ((h << np.uint16(8)) | l).astype(np.uint16)


def words_to_f64(words, dtype):
    """Value of 16-bit words of the given native datatype, as float64 (exact).

    bf16 is the top half of an IEEE binary32; fp16 is IEEE binary16.  Both
    widen exactly to float64.
    """
    w = np.asarray(words, dtype=np.uint16)
    with np.errstate(invalid="ignore"):          # signalling-NaN patterns widen to NaN
        if dtype == "bf16":
            return (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
        if dtype == "fp16":
            return w.view(np.float16).astype(np.float64)
    raise ValueError(f"unsupported dtype {dtype!r}")


def base_value(words, dtype):
    """Value at which a TARGET word is executed once demoted to BASE."""
    return words_to_f64(base_word(hi_byte(words)), dtype)
