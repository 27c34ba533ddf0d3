"""Float64 CPU oracle for the BGPO masked-diffusion ELBO head.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, the smoke check in
``__graft_entry__.py`` and the CPU-baseline leg of ``bench.py`` may import or
run anything in this package.  It shares no code with the HIP path and never
imports it; the two meet only on the seeded inputs of ``workloads``.

Modules:
  philox  Philox4x32-10 and the timestep / mask draws built on it
  elbo    the per-sample ELBO, the lower-bound term, the loss and its
          gradients, in a literal per-sample form and a collapsed form for
          hidden states shared across samples

Parity status: every function here is pinned by the CPU tests
(known-answer vectors, closed forms, brute force, library routines, finite
differences, autograd and the paper's equivalence property).
"""
from . import philox, elbo  # noqa: F401
