"""CPU oracle of the Partial FC head step (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may import
this package.  It shares no code with the HIP path.
"""
from . import philox, pfc_oracle  # noqa: F401
