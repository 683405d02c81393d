"""fp64 CPU oracle of the Jacap scoring path.

TEST INFRASTRUCTURE ONLY: imported by the tests, the package smoke check and
the benchmark's CPU-baseline leg, never by the product path.
"""

from . import jacap_oracle, theory  # noqa: F401
from .jacap_oracle import DIAG, FULL, evict_unit, score_unit, select_top, to_fp32  # noqa: F401
