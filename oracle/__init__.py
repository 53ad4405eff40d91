"""CPU oracle for the LAM hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct implementation of what the GPU library
computes, written from the paper (LAM: A Lossy Agent Memory Framework With a
Retrieval-Score Error Bound):

  * ``oracle.qeps``  -- the quantizer Q_eps(x) = round(x / 2 eps) of Section 2.2
    ("Three layers", L1), its code width and bit packing, decode, and the
    per-element bound;
  * ``oracle.dedup`` -- the epsilon error-bounded test of Algorithm "admit"
    (Section 2.3) with exhaustive candidates, the exact l2 predicate of
    Eq. (identity) (Section 2.1), greedy first-occurrence with the lowest-index
    representative (Appendix "Representative selection"), and the measured
    bound delta_hat (Appendix "The measured bound");
  * ``oracle.score`` -- retrieval scores against the dequantized store, top-k,
    and the Hoelder bound eps*||q||_1 (Appendix "Rank invariance, in full");
  * ``oracle.invariants`` -- checkers for the paper's theorems (Theorem "Score
    deficit", Proposition "greedy is simultaneously a cover and a packing").

Floating point is binary64; every decision that floating point could get wrong
near a tie is re-taken in exact rational (or exact integer) arithmetic.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
and imports nothing from it.
"""
from . import qeps, dedup, score, invariants  # noqa: F401
