"""CPU oracle for the RheoSampling hot path (arXiv 2609.21827).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links anything in this package: only the test-suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.  It
shares no code with the HIP library (no kernels, headers, helpers, tables or
constants); the only thing both sides consume is the seeded synthetic input
generator, which lives in its own module and holds none of the method's
arithmetic.

Layout
  philox.py    Philox4x64-10 counter-based generator (Salmon et al., SC'11)
               and the counter layout used for the method's random draws.
  numerics.py  the two number models: the canonical integer weights that
               take every sampling / acceptance decision, and an fp64 model
               used for the theory pins.
  rheo.py      the method itself, in the paper's order: node distributions,
               the hybrid candidate pool with proxy / true probabilities
               (Sec. 3.2, App. C.1), EAGLE expand-then-rerank (Sec. 2.1),
               global top-R pruning with the tie-breaking rule (App. C.1),
               and RheoVerification (Algorithm 1) run layer by layer
               (Thm. 1).  Random choices are requests yielded by a Python
               generator, so the same code is driven either by Philox draws
               (parity runs) or by exhaustive enumeration (theory pins).
  drivers.py   the Philox driver and the exact-enumeration driver.
"""
