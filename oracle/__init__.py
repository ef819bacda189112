"""CPU oracle for the DCP hot path (test infrastructure, not product code).

Only the test suite, the smoke check in ``__graft_entry__`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.
The GPU path never calls it and shares no code with it.

Modules
-------
attention : float64 numpy block-diagonal (packed) exact self-attention,
            forward and analytic backward, plus row-sampled variants.
planner   : Python-int DCP planner (DCP-intra, DCP-inter, gradient
            accumulation search) and exhaustive brute-force searches.
"""
