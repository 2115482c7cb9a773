"""fp64 CPU oracle for the LoSA hot path -- test infrastructure only.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package; the product path (paper_2608_12032_amd) never does.
"""
from . import losa_oracle, compare  # noqa: F401
