"""CPU float64 oracle of the W4+EC linear layer (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package. The product path (paper_2606_11244_amd) never does.
"""
from . import spear_oracle  # noqa: F401
