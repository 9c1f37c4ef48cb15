"""CPU oracle for PETRA's per-stage reversible step (test infrastructure only).

This package is a plain, slow, obviously correct numpy implementation of what
the hot path computes.  It exists to check the HIP path and nothing else:
only the test-suite, the smoke check and the CPU-baseline leg of the benchmark
may import it.  The product path never calls into it, and it imports nothing
from the product package (no shared kernels, helpers, tables or constants).

Default arithmetic is fp64.  Every function cites the passage of the paper it
follows; where the paper is silent the chosen reading is stated in place.

Pins (tests/test_oracle_*.py) tie it to things other than itself:
  * conv / BN / ReLU forward and VJP against torch CPU autograd in fp64 and a
    brute-force loop on tiny shapes;
  * inverse(forward(x)) == x with frozen parameters (Eq. 4);
  * frozen-parameter reconstruct+VJP == ordinary backprop (Eqs. 2-4);
  * central finite differences on tiny inputs;
  * BN invariants, the identity-block special case, SGD closed forms,
    gradient-accumulation averaging (Alg. 1), and the tick table of the
    multi-stage schedule (delay 2(J-j), App. B).
Parity unpinned: the stale-parameter reconstruction of Eq. (5) when the
parameters change between a forward and its backward has no closed form; it is
pinned only through its frozen-parameter special case and the step order.
"""
from . import conv, bn, revblock, stage, sgd  # noqa: F401
