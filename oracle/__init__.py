"""CPU oracle for the FreqCache hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct reference implementations (numpy) of
cacheable-token selection (float64) and the partial-recompute decoder layer
(float32).  Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
leg may import anything here; the product path (paper_2604_24391_amd) never
does and shares no code with it.

Parity pins: every function is pinned by tests/test_oracle_*.py against
library routines, closed forms, invariants and brute force (see each test's
docstring).  The paper prints no worked numeric example, so the readings
where it is silent (see the select and layer module headers) rest on those
pins and on the paper's hyper-parameters, not on printed intermediate values.
"""
from . import select, layer  # noqa: F401
