"""CPU oracle of RaBitQCache's decode path: test infrastructure only.

Only tests/, the package smoke check and bench.py's CPU-baseline leg may use
it; the HIP library never does.
"""
from . import rbq_oracle  # noqa: F401
