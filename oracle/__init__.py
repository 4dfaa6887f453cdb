"""CPU oracle for the verify-block MoE layer (test infrastructure only)."""
from . import acceptmoe_oracle  # noqa: F401
