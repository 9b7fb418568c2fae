"""Plain, slow CPU oracle for the ElasticKV mixed-fidelity KV hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only the test-suite, the package's smoke check and the
``cpu_baseline`` leg of the benchmark use it.  It shares no code with the HIP
library (no kernels, headers, helpers, tables or pre/post-processing); it
operates on plain NumPy arrays handed to it by the caller.

What it computes, and where the paper defines it:

* ``encoding``   -- TARGET is the native 16-bit KV word, BASE keeps its
  high-order 8 bits, the low-order 8 bits refine BASE exactly (§3, opening
  paragraph; App. B.2).  BASE is consumed by placing the byte back in the
  high-order position with a zero low byte (§3.2; App. B.3).
* ``paged``      -- logical-to-physical gather through a block table
  (§2.1), with the pair-structured layout of §3.1.
* ``attention``  -- softmax attention for decode and chunked prefill over a
  mixed TARGET/BASE sequence (§3.2), in float64.
* ``transitions``-- demotion (pack a TARGET pair into one block, free the
  other), refinement (restore the pair exactly, reacquire one block),
  append of new TARGET KV, and the free-block FIFO (§3.1; §3.4; App. B.2).
* ``lowering``   -- batch-level BASE indicator, per-sequence TARGET-BASE-
  TARGET boundaries or an explicit pair-mode table (§3.2; App. B.3).
* ``validate``   -- the metadata invariants those steps rely on (pairs share
  one fidelity, BASE pairs are two full blocks in one physical block,
  transitions start from the opposite state; §3.1, App. B.1).
* ``control``    -- the pressure-aware fidelity controller: shortage,
  demotion count, surplus, decaying reserve and promotion budget, with the
  rank orders of its candidates (§3.3, Alg. 1; App. B.1).
* ``fp8``        -- the 8-bit TARGET (E5M2) / 4-bit BASE instance of the
  same contract: encoding, packed nibble pairs, transitions, decode and
  prefill (App. C.5, last paragraph).

Readings of points the paper leaves open (pair membership, which block of a
pair survives demotion, the byte layout inside a packed block, where the
refinement bytes live, allocator order, the softmax scale, the GQA head map)
are stated in the docstrings of the functions that take them.

Parity status: every function here is pinned by tests that do not re-type its
formula (closed forms, exhaustive enumeration, brute force on tiny inputs,
library routines, invariants); see the ``tests/test_oracle_*.py`` files.
"""

from . import encoding, paged, attention, transitions, lowering, validate, control, fp8  # noqa: F401
