"""CPU oracle (test infrastructure only; see int2kv_oracle)."""
from . import int2kv_oracle  # noqa: F401
