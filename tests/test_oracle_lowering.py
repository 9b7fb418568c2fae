"""Pins for oracle.lowering: the structured/general split of §3.2 checked
against a regular expression over pair-mode strings, and boundaries checked
by rebuilding the tag table from them."""

import re

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import lowering

PAGE = 16


def _tags_from_modes(modes, max_blocks):
    row = np.zeros(max_blocks, dtype=np.uint8)
    for j, m in enumerate(modes):
        row[2 * j] = row[2 * j + 1] = m
    return row


@settings(max_examples=300, deadline=None)
@given(st.lists(st.lists(st.integers(0, 1), min_size=1, max_size=12), min_size=1, max_size=6),
       st.integers(0, 31))
def test_lowering_matches_regex_and_rebuilds_tags(mode_lists, tail):
    max_blocks = 2 * max(len(m) for m in mode_lists) + 2
    tags = np.stack([_tags_from_modes(m, max_blocks) for m in mode_lists])
    seq_lens = np.array([2 * PAGE * len(m) for m in mode_lists], dtype=np.int32)
    mode, bounds = lowering.lower(tags, seq_lens, PAGE)
    strings = ["".join("B" if x else "T" for x in m) for m in mode_lists]
    any_b = any("B" in s for s in strings)
    regular = [re.fullmatch(r"T*B*T*", s) is not None for s in strings]
    if not any_b:
        assert mode == lowering.NATIVE
    elif all(regular):
        assert mode == lowering.STRUCTURED
    else:
        assert mode == lowering.GENERAL
    for s, m in enumerate(mode_lists):
        b0, b1 = bounds[s]
        if regular[s]:
            rebuilt = [1 if b0 <= j < b1 else 0 for j in range(len(m))]
            assert rebuilt == list(m)
        else:
            assert (b0, b1) == (-1, -1)


def test_invisible_blocks_are_ignored():
    tags = np.zeros((1, 8), dtype=np.uint8)
    tags[0, 6:] = 1                      # past the end of a 40-token sequence
    mode, bounds = lowering.lower(tags, np.array([40]), PAGE)
    assert mode == lowering.NATIVE and tuple(bounds[0]) == (0, 0)
