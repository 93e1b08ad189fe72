"""CPU oracle for the Random Attention decode hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only the tests, the smoke check of
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.  It
shares no code with the HIP path; the two meet only through the seeded
workload generator, which holds none of the method's arithmetic.

Everything here is plain numpy (fp64 for floating point, uint64 for the
random keys) and follows the paper's statement of the method:

* ``philox``    -- the counter-based generator that supplies the per-head
                   uniform draws (reading of the per-request seed).
* ``evict``     -- the eviction rule: candidate set, uniform scores with the
                   prompt at +infinity, top-K keep set (Eq. 1, Section 3,
                   Appendix F), and an index-only replay of a whole decode.
* ``attention`` -- exact softmax GQA decode attention over the kept rows
                   (Section 2, "Notation").
* ``decode``    -- the full decode loop (append, attend, periodic evict) for
                   the small cases the oracle finishes in seconds.

Parity status of each function is stated in its module header.
"""

from . import philox, evict, attention, decode  # noqa: F401
