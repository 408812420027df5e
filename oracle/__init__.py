"""CPU fp64 oracle (test infrastructure only; see gp_oracle's module docstring)."""
from . import gp_oracle  # noqa: F401
