"""Plain, slow, obviously-correct CPU oracle for Geodesia-KV graded decode attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it.  It shares no code with the HIP library (no kernels, no
headers, no layout tables); the two meet only through the seeded input
generators, which hold none of the method's arithmetic.

Everything is numpy in float64.  Results that the GPU must reproduce bit for bit
(quantized codes, scales, zeros, centroids, ids, page boxes, Quest page sets and
residual token sets) are written with explicit sequential loops over every
reduction axis, one IEEE rounding per operation and no fused multiply-add, so the
order of operations is part of the definition.  Attention outputs are computed in
any order and compared under a tolerance.

Modules (each cites the passage of the paper it follows):

* ``fp16``        -- fp16 <-> fp64 conversions (single round-to-nearest-even).
* ``ladder``      -- the age-ordered monotone precision ladder (Method, section 3.2).
* ``quant``       -- block scalar quantizer, centroid state, demotion (section 3.2).
* ``quest``       -- exact per-page key boxes and box upper-bound ranking (section 3.5).
* ``attention``   -- single-query GQA decode attention over a graded read set
                     (sections 3.5 and 3.7).
* ``residual``    -- rate-distortion exact residual selection (section 3.4, Eq. rdscore).
* ``accounting``  -- resident / read bits per value (section 3.5 rate equations,
                     section 4.4 metrics).
* ``certificate`` -- the attention error certificate (section 3.6, Eq. certificate),
                     used as an independent pin on the attention oracle.
* ``cache``       -- a whole graded cache for one (sequence, KV head) unit built
                     from the functions above.

Parity status: every function above is pinned by tests in ``tests/`` against
closed forms, invariants, brute force, or values printed in the paper, except
where a function's docstring says "parity unpinned".
"""

from . import fp16, ladder, quant, quest, attention, residual, accounting, certificate, cache  # noqa: F401
