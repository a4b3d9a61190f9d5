"""Plain CPU oracle for the HilbertA hot path (HilbertA, arXiv 2509.26538).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  The HIP library never
falls back to it.

Everything here is slow and obviously correct on purpose:

* ``hilbert``    -- the Hilbert linearisation pi of a 2^k x 2^k grid (§3.1),
                    built twice, by the iterative bit-pair algorithm and by an
                    L-system turtle, so that each pins the other; other grid
                    shapes embedded in their enclosing 2^k square with padding
                    (Appendix D).
* ``schedule``   -- tile labels, sliding offsets, the central shared region,
                    the explicit 0/1 attention mask (§3.2, §3.3, Appendix A)
                    and the schedule table in the library's documented layout.
* ``attention``  -- masked softmax attention in float64 from its closed
                    form, plus a pure-Python loop version for tiny inputs.
* ``gradients``  -- dQ, dK, dV of the masked attention by the chain rule
                    (the backward pass training needs).
* ``tokens``     -- the token gather / scatter of §3.4.
* ``accounting`` -- nnz of the mask and the FLOP count of §4.2.

No function shares code, tables or constants with the HIP path; the two meet
only on seeded inputs produced elsewhere.
"""

from . import hilbert, schedule, attention, gradients, tokens, accounting  # noqa: F401
