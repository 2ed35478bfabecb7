"""CPU oracle for the ASAP hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct NumPy (fp64) statement of what one ASAP round
computes: each worker's local minibatch SGD half-step followed by the
stochastic reduce over a doubly-stochastic communication graph (Appendix A,
update equation (A.2); the mixing matrix P of the "Network requirement"
paragraph), plus the graph builders, the sample schedule and the per-round
metrics that the hot path relies on.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import anything from this package.  It shares no code with the HIP library:
the two sides meet only in the seeded input generators, which hold none of the
method's arithmetic.

Parity status of each function is stated in its module header; a function with
no independent pin says "parity unpinned".
"""
from . import prng, graphs, sgd, mix, metrics, rounds  # noqa: F401,E402
