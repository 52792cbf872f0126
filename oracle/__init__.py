"""CPU oracle of the DPara drafter hot path (test infrastructure only).

Only tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package.  The product package never does."""
from . import dpara_oracle  # noqa: F401
