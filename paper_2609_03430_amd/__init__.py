"""Random Attention decode hot path for MI355X (gfx950).

Per-KV-head compressed KV cache: the prompt and the r most recent tokens are
always kept, the remaining entries are evicted uniformly at random down to a
budget of K per head, with no scoring pass.  The work is done by hand-written
HIP kernels behind the C ABI declared in ``include/randattn.h``; ``binding``
marshals torch tensors and streams into those calls.  ``synth`` produces the
seeded synthetic inputs used by tests and the benchmark.

Importing the package loads nothing; ``binding`` loads the shared library on
first use and raises if it is missing.
"""
