"""CPU oracle for the SSD verify step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct numpy implementation (float64 arithmetic) of
what the batched verify step of Spatially Speculative Decoding computes:

* ``model``    -- the frozen decoder-only backbone forward pass with a KV cache
                  (Sec. 3.1, Eq. 1: raster-order autoregressive image tokens),
                  and the block ("verification") forward of Sec. 3.3.
* ``select``   -- the three per-position correction rules (A) greedy,
                  (B) sampling, (C) acceptance-rejection with the residual
                  distribution, and the counter-based uniform generator.
* ``decode``   -- verify rounds, the commit pass, strict truncation
                  (exact speculative decoding), greedy AR decoding and the
                  whole-image schedule (horizontal stage + vertical rows).
* ``schedule`` -- the pass plan of an image (k_h, horizontal rounds, k_v, b, i).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
(``paper_2606_20543_amd``) and never imports it; the only module both sides
use is the seeded input generator ``synth``, which holds none of the method's
arithmetic.

Pins (what each function is checked against) are listed in each module's
docstring; anything not pinned says "parity unpinned".
"""

from . import select, model, schedule, decode  # noqa: F401
