"""TEST INFRASTRUCTURE ONLY -- the plain CPU oracle of BASE's decode hot path.

Written from the paper, independent of the HIP library: it shares no code,
headers, tables or helpers with ``paper_2609_36222_amd`` and neither imports
the other.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may use it; the product path never does.

* ``carith``  -- canonical fp32 arithmetic (C, exact single-rounding FMA):
                 cexp, fixed-order dot, router, predictor, aggregation, gates.
* ``method``  -- fp64 definitions of the paper's quantities, the integer
                 selection / backfill / compaction logic, diagnostics.
* ``calib``   -- ridge calibration of the log-energy predictor (App. A).
"""
from . import carith, method, calib  # noqa: F401
