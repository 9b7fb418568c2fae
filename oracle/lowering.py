"""Dual-mode dispatch metadata (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

§3.2 and App. B.3: a batch-level indicator sends TARGET-only batches to the
native path and batches holding any BASE block to the elastic path.  Inside
the elastic path each sequence's attention-visible KV is an ordered
sequence of pair modes.  A sequence of the form TARGET* BASE* TARGET* (at
most two mode boundaries) is described by its boundaries and takes the
structured path; any other sequence carries an explicit pair-mode table and
takes the general path.

Encoding used here:

* ``mode`` -- NATIVE if no visible block is BASE; STRUCTURED if every
  sequence is TARGET* BASE* TARGET*; GENERAL otherwise;
* ``boundaries[s] = (b0, b1)`` in pair units: pairs ``b0 <= j < b1`` are BASE
  and all other pairs TARGET (``b0 == b1`` means no BASE pair); an irregular
  sequence gets ``(-1, -1)`` and is served from the tag table.

Only blocks that hold tokens (``ceil(L/page)`` of them) are visible; table
entries beyond them are ignored.
"""

import numpy as np

NATIVE = 0
STRUCTURED = 1
GENERAL = 2


class InvalidTags(ValueError):
    """Tags that differ between the two members of a pair."""


def pair_modes(tag_row, length, page):
    """Mode of each pair that holds at least one visible block."""
    nblk = -(-int(length) // page)
    modes = []
    for j in range((nblk + 1) // 2):
        a = int(tag_row[2 * j])
        b = int(tag_row[2 * j + 1]) if 2 * j + 1 < nblk else a
        if a != b:
            raise InvalidTags(f"pair {j} has mixed tags")
        modes.append(a)
    return modes


def lower(tags, seq_lens, page):
    """Return (mode, boundaries int32 [B][2])."""
    bsz = len(seq_lens)
    bounds = np.zeros((bsz, 2), dtype=np.int32)
    any_base = False
    any_irregular = False
    for s in range(bsz):
        modes = pair_modes(tags[s], seq_lens[s], page)
        base_pairs = [j for j, m in enumerate(modes) if m != 0]
        if not base_pairs:
            bounds[s] = (0, 0)
            continue
        any_base = True
        b0, b1 = base_pairs[0], base_pairs[-1] + 1
        if all(modes[j] != 0 for j in range(b0, b1)):
            bounds[s] = (b0, b1)
        else:
            bounds[s] = (-1, -1)
            any_irregular = True
    if not any_base:
        return NATIVE, bounds
    return (GENERAL if any_irregular else STRUCTURED), bounds
