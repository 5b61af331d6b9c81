"""CPU oracle of the integer training dataflow of arXiv 2011.14504.

TEST INFRASTRUCTURE ONLY.  A plain, slow, exact implementation (C with
__int128 in iseg_oracle.c, composed in oracle.py) of the paper's quantizers
(Eq. 1-6), weight/update quantizers (Eq. 7, 8, 19), integer convolutions, the
square/root-free L1 batch normalization (Eq. 12-15) and its backward, and the
max-pool glue.  Only tests/, __graft_entry__.smoke() and bench.py's CPU
baseline may import it; the GPU library never does, and the two share no code.

Pins (tests/test_oracle_*.py) tie it to the paper and to mathematics other than
itself: hand-worked examples (tests/golden/), exact-rational brute force of the
paper's real-valued formulas, float64 library convolutions, the adjoint
identity, finite differences of Eq. 12-13, the Philox known-answer vectors and
statistical unbiasedness of Eq. 6.

Parity unpinned: the L1BN backward composition.  The paper prints no formula
or value for it; the oracle uses the exact derivative of Eq. 12-13 with
straight-through quantizers, which is pinned only against finite differences
and the exact-rational brute force of that same reading.
"""
