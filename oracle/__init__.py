"""CPU float64 oracle (test infrastructure only; see fq_oracle)."""
from .fq_oracle import *  # noqa: F401,F403
