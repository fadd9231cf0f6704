"""Plain CPU oracle for the fully-quantized-training (FQT) layer backward.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no headers, helpers, tables or constants).

Every function follows a passage of Chen et al., "A Statistical Framework for
Low-bitwidth Training of Deep Neural Networks" (NeurIPS 2020), cited by section
and equation.  Floating point is numpy float64 unless the determinism contract
below fixes a float32 step; those float32 steps are single IEEE operations in a
stated order, which numpy evaluates without contraction.

Determinism contract (shared by definition, not by code, with the GPU path):

* stochastic rounding draws come from Philox4x32-7 (``philox.py``), keyed by
  the seed, with the element's logical row-major index as counter;
* per-tensor / per-sample / block-Householder scales and zero points are
  computed by the formulas in ``quantizers.py``;
* integer accumulators are exact (int64 here).

Modules:
  philox      -- Philox4x32 counter-based generator (Salmon et al., SC'11), 7 rounds
  sr          -- stochastic rounding SR(.) of Sec. 3.3 and its exact moments
  quantizers  -- PTQ (Sec. 3.3), PSQ (Sec. 4.1), BHQ (Sec. 4.2, App. C.4, App. D)
  backward    -- linear / conv layer backward of Sec. 2.2 (Eq. linear-sq-backprop)
  theory      -- closed forms used as pins (App. B, App. C)
"""
