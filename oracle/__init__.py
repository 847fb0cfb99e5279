"""CPU oracle of the single-stage forward -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may import this package.  The product (``paper_2512_21835_amd``) never does,
and this package imports nothing from the product: the two share no code.  Both
read their inputs from ``synth`` (shapes, seeds, random numbers only).

* ``stage_oracle``: plain float64 numpy definition of the stage forward.
* ``policies``: independent re-implementations of the integer policies (paged
  KV block allocation, slot assignment of streamed layers, residency schedule)
  whose results the HIP runtime must reproduce bit-exactly.
* ``planner``: the online memory-aware planner (Eq. (7)) by brute force over
  every (alpha, beta), one token count at a time.
"""
from . import stage_oracle, policies, planner  # noqa: F401
