"""CPU oracle for DLM-based lossless compression -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct fp64 NumPy implementation of the masked
diffusion compression step of "Diffuse to Compress" (Nardone & Ferragina):

* ``weights``  -- the counter-based random init of every tensor
* ``model``    -- the masked diffusion LM forward pass (Definition 3)
* ``schedule`` -- per-position entropy and the entropy-based commitment
                  schedule (Symbol Commitment Schedules, item 3)
* ``cdf``      -- quantisation of a predicted distribution into an integer CDF
                  for the statistical coder (Implementation Details: rANS /
                  statistical coding of each committed symbol)
* ``coder``    -- a carry-propagating range coder
* ``driver``   -- the iterative pipeline of Section "Diffusion-Based
                  Compression Pipeline": S(0) = all MASK, repeat forward ->
                  schedule -> encode -> reveal

It shares no code with the HIP path.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import it;
the product library never calls it.
"""
from . import weights, model, schedule, cdf, coder, driver  # noqa: F401
