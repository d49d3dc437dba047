"""CPU float64 oracle for HeadCast routed attention (test infrastructure only:
imported by tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg)."""
from .headcast_oracle import *  # noqa: F401,F403
